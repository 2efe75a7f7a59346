/*
 * gnnprop -- GraphSAGE feature propagation on a sampled subgraph, forward
 * and backward, on AMD Instinct MI355X (gfx950).
 *
 * The operations follow "Accurate, Efficient and Scalable Training of Graph
 * Neural Networks" (Zeng, Zhou, Srivastava, Kannan, Prasanna):
 *   - one layer's forward, Section 2.1, Eq. "graphsage forward":
 *       Y = ReLU( X W_self || A_s X W_neigh )      (self half first)
 *     with A_s the subgraph's normalised adjacency (D^-1 A for GraphSAGE);
 *   - its backward, Section 5.1, Eq. "gcn backward";
 *   - the three kernels Section 5.1 names: sparse feature / gradient
 *     propagation (CSR SpMM), dense weight transformation (GEMM on the
 *     matrix cores), and the sparse adjacency transpose (Section 5.2,
 *     Algorithm 6);
 *   - the computation-order choice of Section 6.1.
 *
 * Conventions for every entry point
 *   - Pointers named as device pointers must point to memory of the current
 *     HIP device; the library never takes ownership and never frees them.
 *   - Dense matrices are row-major fp32 with an explicit leading dimension
 *     (row stride, in elements, >= the row width).  Any 4-byte-aligned
 *     pointer and any stride is accepted; 16-byte alignment of the base and a
 *     stride that is a multiple of 4 enable the vector paths.
 *   - Work is enqueued on `stream` (NULL = the null stream) and is complete
 *     once the stream is synchronised.  Only gnn_csr_validate synchronises.
 *   - Argument errors are reported synchronously, before anything is
 *     enqueued; a failed launch returns GNN_ERR_HIP.  Nothing is printed and
 *     no C++ exception crosses this interface.
 *   - Outputs are overwritten, never accumulated into.  Inputs and outputs
 *     must not overlap unless an entry point says otherwise.
 *   - gnn_prop_fwd / gnn_prop_bwd / gnn_spmm / gnn_gemm allocate no device
 *     memory: scratch comes from the caller's `workspace`.
 *   - `workspace`, `saved` and plan buffers (csr->plan included) must start
 *     16-byte aligned, as hipMalloc memory does; any other address is
 *     GNN_ERR_UNSUPPORTED.
 */
#ifndef GNNPROP_H
#define GNNPROP_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum gnn_status {
  GNN_OK = 0,
  GNN_ERR_NULL = -1,        /* a required pointer is NULL */
  GNN_ERR_SHAPE = -2,       /* a size or leading dimension is invalid */
  GNN_ERR_CSR = -3,         /* gnn_csr_validate found an invalid CSR */
  GNN_ERR_UNSUPPORTED = -4, /* option not supported */
  GNN_ERR_WORKSPACE = -5,   /* workspace or plan buffer too small */
  GNN_ERR_HIP = -6,         /* a HIP runtime call or launch failed */
  GNN_ERR_ALIAS = -7        /* outputs overlap inputs where forbidden */
} gnn_status;

/* Layer flags. */
/* GEMM products.  By default every fp32 operand of a weight transformation
 * is split exactly into three bf16 pieces (x = hi + mid + lo, each rounded
 * to nearest even) and the six piece products down to 2^-16 of hi x hi are
 * accumulated in fp32 on the bf16 matrix cores: fp32 operands, results and
 * accumulation, with a product error below 2^-24 relative (measured against
 * fp64: no larger than that of the fp32 matrix-core instruction).  Operands
 * must be finite and below bf16's largest finite value (about 3.39e38) in
 * magnitude: an infinite operand makes its outputs NaN where the fp32
 * instruction gives infinities (use GNN_FLAG_F32_MFMA for such data).  The
 * two flags below select other arithmetic; setting both is
 * GNN_ERR_UNSUPPORTED. */
#define GNN_FLAG_BF16 0x1u /* GEMM operands rounded to bf16 (round to nearest
                              even), fp32 accumulation; the aggregation sums
                              in fp32 (in the backward pass its output T and
                              the mask's G_s are kept in the workspace already
                              rounded, as only the GEMMs read them); all
                              outputs fp32 */
#define GNN_FLAG_F32_MFMA 0x8u /* GEMM products on the fp32 matrix-core
                                  instruction (v_mfma_f32_32x32x2_f32) */
/* GraphSAGE layers only (gnn_prop_fwd / gnn_prop_bwd).  Section 2.1 defines
 * the layer's A_s as D^-1 A, D the diagonal of A's row sums; with this flag
 * the aggregations take A_s from the pattern alone, A the 0/1 matrix of the
 * stored entries (self loops as stored) and deg(v) = indptr[v+1] - indptr[v]:
 * the forward sums each row's neighbour rows unweighted and scales the sum
 * by 1/deg(v), the transposed aggregation weighs entry (u, v) by 1/deg(v)
 * (the value (A_s)^T holds there when the pattern is symmetric, as the
 * backward pass requires anyway).  csr->values and csr->values_t are then
 * not read and may be NULL.  Results equal those of the same call with
 * values = 1/deg in float (values_t from gnn_csr_transpose_values) up to
 * rounding: the forward rounds the sum before the scaling. */
#define GNN_FLAG_ROW_NORMALIZED 0x10u
/* Backward pass only (Algorithm 1's layer loop, backward direction): the
 * layers of a stack share their ReLU masks.  Layer l's input X is layer
 * l-1's output, so 1[X > 0] is layer l-1's mask and can be applied where
 * layer l produces dX; layer l-1 then receives its G directly. */
#define GNN_FLAG_DY_MASKED 0x2u /* dY is already G = dY * 1[Y > 0]: no
                                   masking pass, dY is read in place */
#define GNN_FLAG_DX_MASKED 0x4u /* dX is written as dX * 1[X > 0] (selected,
                                   not multiplied), i.e. the next layer
                                   down's G when X is that layer's output */

/* The sampled subgraph's adjacency A_s in CSR (Section 5.2: Indptr,
 * Indices, Data).  All arrays are device memory.
 *   indptr  [n+1]  indptr[0] = 0, non-decreasing, indptr[n] = nnz
 *   indices [nnz]  column ids in [0,n), ascending within each row
 *   values  [nnz]  A_s entries (any values; D^-1 A for GraphSAGE)
 *   values_t[nnz]  entries of (A_s)^T on the same indptr/indices, from
 *                  gnn_csr_transpose_values; needed by the backward pass
 *                  and by gnn_spmm with transpose = 1.  The transpose reuses
 *                  indptr/indices, so the pattern must be symmetric
 *                  (undirected subgraph, Section 5.2).
 *   plan           device buffer written by gnn_csr_build_plan (or
 *                  gnn_csr_prepare): per window of 256 stored entries the
 *                  rows whose first entry lies in it and their entry range,
 *                  and the row of every entry. */
typedef struct gnn_csr {
  int32_t n;
  int64_t nnz;
  const int32_t* indptr;
  const int32_t* indices;
  const float* values;
  const float* values_t;
  const void* plan;
} gnn_csr;

/* One layer's shape.  X is n x f_in (stride ld_x); Y and dY are n x 2h
 * (stride ld_y), self half in columns [0,h), neighbour half in [h,2h);
 * dX is n x f_in (stride ld_dx); W_self and W_neigh are f_in x h, dense
 * row-major (stride h); biases are [h].
 *   order: 0 = choose by gnn_choose_order, 1 = (A_s X) W_neigh,
 *          2 = A_s (X W_neigh).  Both orders compute the same values. */
typedef struct gnn_layer {
  int32_t f_in;
  int32_t h;
  int64_t ld_x;
  int64_t ld_y;
  int64_t ld_dx;
  int32_t order;
  uint32_t flags;
} gnn_layer;

/* Human-readable name of a status code (static storage). */
const char* gnn_status_string(gnn_status s);

/* Section 6.1: for A (sparse n x n) . W1 (n x f1) . W2 (f1 x f2), order 1
 * (A W1) W2 costs delta n^2 f1 + n f1 f2 multiply-adds and order 2
 * A (W1 W2) costs delta n^2 f2 + n f1 f2.  Returns 1 when f1 <= f2 (ties go
 * to order 1), else 2.  For a layer, f1 = f_in and f2 = h. */
int32_t gnn_choose_order(int32_t f_in, int32_t h);

/* ---------------------------------------------------- per-subgraph prep */

/* Section 5.2, Algorithm 6: values of (A_s)^T on the pattern of A_s.  For
 * each stored (v,u), writes values[pos(v,u)] to values_t[pos(u,v)]; a pure
 * permutation, bit-exact.  Requires csr->indptr/indices/values; the pattern
 * must be symmetric with ascending indices per row (check with
 * gnn_csr_validate).  values_t is device memory of nnz floats.  If
 * csr->plan is non-NULL it must hold this graph's plan (gnn_csr_build_plan,
 * enqueued before), whose per-entry rows then give one thread to each
 * entry; with plan == NULL one wavefront handles each row. */
gnn_status gnn_csr_transpose_values(const gnn_csr* csr, float* values_t,
                                    hipStream_t stream);

/* Bytes of the aggregation work plan for a graph of n rows and nnz entries. */
size_t gnn_plan_bytes(int32_t n, int64_t nnz);

/* Builds the aggregation work plan into `plan` (device memory of at least
 * gnn_plan_bytes(n, nnz) bytes).  The stored entries are cut into windows of
 * 256; window k gets the rows whose first entry lies in it (so a row, hub
 * rows included, is never shared between windows) and their entry range,
 * and every entry its row.  The aggregation gives each window to one
 * workgroup and splits its entries evenly over lane groups; the parts of a
 * row cut between groups are added in a fixed order, so results are
 * deterministic.  Reads csr->n, nnz and indptr. */
gnn_status gnn_csr_build_plan(const gnn_csr* csr, void* plan,
                              size_t plan_bytes, hipStream_t stream);

/* Both per-subgraph preparations (Section 5.2) in one launch: the plan of
 * gnn_csr_build_plan into `plan` (plan_bytes >= gnn_plan_bytes) and the
 * transposed values of gnn_csr_transpose_values into values_t (nnz floats).
 * The results are bit for bit those of the two separate calls.  The
 * pattern must be symmetric with ascending indices per row; csr->values_t
 * and csr->plan are not read.  plan and values_t may not overlap each
 * other or the CSR arrays (GNN_ERR_ALIAS). */
gnn_status gnn_csr_prepare(const gnn_csr* csr, void* plan, size_t plan_bytes,
                           float* values_t, hipStream_t stream);

/* Checks the CSR on the device and synchronises `stream`: indptr
 * monotone with indptr[0] = 0 and indptr[n] = nnz, indices in range and
 * strictly ascending per row, and, if require_symmetric, that every stored
 * (v,u) has a stored (u,v).  Returns GNN_OK or GNN_ERR_CSR.  May allocate a
 * few bytes of device memory. */
gnn_status gnn_csr_validate(const gnn_csr* csr, int32_t require_symmetric,
                            hipStream_t stream);

/* gnn_csr_validate for callers that cannot allocate device memory (serving
 * loops, harnesses that forbid hipMalloc): the same checks and the same
 * result, with the status word the check writes kept in a 256-byte array
 * of static device memory that the library holds on each device it runs on
 * until the process ends, instead of a hipMalloc'd word.  That scratch does
 * not grow with the graph, so no size limit applies beyond those of
 * gnn_csr_validate.  Every call on one device shares the array (each call
 * clears it first): calls that overlap on one device race and must be
 * serialised by the caller.  Synchronises `stream`; calls no hipMalloc or
 * hipFree. */
gnn_status gnn_csr_validate_noalloc(const gnn_csr* csr,
                                    int32_t require_symmetric,
                                    hipStream_t stream);

/* ------------------------------------------------------------ one layer */

/* Device bytes the forward pass saves for the backward pass, and the
 * scratch bytes forward and backward need.  Order 1 saves A_s X (n x f_in
 * floats).  With split products (neither product flag) the forward's weight
 * split also writes the bf16 pieces of W_self^T and W_neigh^T that the input
 * gradient's product uses (3 x 2 x ceil(h / 16) x 16 x f_in bytes each), so
 * that the backward pass does not split the weights again; with
 * GNN_FLAG_BF16 or GNN_FLAG_F32_MFMA order 2 saves nothing.  Both sizes
 * depend only on csr->n, csr->nnz, the layer shape, its order and its
 * product flag. */
size_t gnn_prop_saved_bytes(const gnn_csr* csr, const gnn_layer* layer);
size_t gnn_prop_workspace_bytes(const gnn_csr* csr, const gnn_layer* layer);

/* Forward of one layer, Section 2.1 Eq. "graphsage forward":
 *   Y[:, 0:h]  = ReLU(X W_self + b_self)
 *   Y[:, h:2h] = ReLU(A_s X W_neigh + b_neigh)
 * b_self / b_neigh may be NULL (no bias: the paper's form).  Needs
 * csr->values and csr->plan.  `saved` (gnn_prop_saved_bytes, may be NULL
 * when that is 0 or csr->n is 0) receives what gnn_prop_bwd needs and must
 * be passed to it unchanged.  Y must not overlap X. */
gnn_status gnn_prop_fwd(const gnn_csr* csr, const gnn_layer* layer,
                        const float* X, const float* W_self,
                        const float* W_neigh, const float* b_self,
                        const float* b_neigh, float* Y, void* saved,
                        void* workspace, size_t workspace_bytes,
                        hipStream_t stream);

/* Backward of one layer, Section 5.1 Eq. "gcn backward", given the forward
 * output Y (its sign pattern is the ReLU mask: G = dY * 1[Y > 0], 0 at the
 * kink) and dY = dL/dY:
 *   dW_self  = X^T G[:, 0:h]
 *   dW_neigh = (A_s X)^T G[:, h:2h]
 *   dX       = G[:, 0:h] W_self^T + (A_s)^T G[:, h:2h] W_neigh^T
 *   db_self, db_neigh = column sums of the two halves of G
 * dX may be NULL (not computed; e.g. the first layer).  db_* may be NULL.
 * layer->flags may add GNN_FLAG_DY_MASKED (dY already masked) and
 * GNN_FLAG_DX_MASKED (dX returned masked by 1[X > 0]) to the product flags
 * (GNN_FLAG_BF16 or GNN_FLAG_F32_MFMA, or neither: split products).
 * Needs csr->values, csr->values_t and csr->plan, and the `saved` buffer of
 * the matching gnn_prop_fwd call with the same layer (same order and product
 * flag) and the same weights: with split products the input gradient takes
 * the weights' pieces saved by that call (as in training, where the
 * backward pass follows the forward pass that used the weights).  Outputs
 * must not overlap inputs. */
gnn_status gnn_prop_bwd(const gnn_csr* csr, const gnn_layer* layer,
                        const float* X, const float* W_self,
                        const float* W_neigh, const float* Y, const float* dY,
                        const void* saved, float* dX, float* dW_self,
                        float* dW_neigh, float* db_self, float* db_neigh,
                        void* workspace, size_t workspace_bytes,
                        hipStream_t stream);

/* ------------------------------------------------- GCN and MixHop layers */

/* The GNN variants of Section 2.1 on the same three kernels; their
 * backward keeps the A_hat terms of the Section 5.1 gradients.
 * csr->values must hold A_hat = (I + D)^-1/2 (I + A) (I + D)^-1/2 (the
 * pattern storing the self loops); it is symmetric, so csr->values_t may
 * point to csr->values.  layer->h is one path's output width; layer->flags
 * may hold one product flag (GNN_FLAG_BF16 or GNN_FLAG_F32_MFMA) only.  Sizes
 * of `saved` and workspace come from the matching queries; ownership and
 * aliasing rules are those of gnn_prop_fwd / gnn_prop_bwd.
 *
 * GCN (Eq. "gcn forward"): Y = ReLU(A_hat X W + b), Y n x h (stride
 * ld_y >= h), W f_in x h row-major, b [h] or NULL; order as for GraphSAGE
 * (1: (A_hat X) W, A_hat X saved; 2: A_hat (X W)).  Backward: G = dY *
 * 1[Y > 0], dW = (A_hat X)^T G, dX = A_hat^T G W^T (dX may be NULL),
 * db = column sums of G (db may be NULL). */
size_t gnn_gcn_saved_bytes(const gnn_csr* csr, const gnn_layer* layer);
size_t gnn_gcn_workspace_bytes(const gnn_csr* csr, const gnn_layer* layer);
gnn_status gnn_gcn_fwd(const gnn_csr* csr, const gnn_layer* layer,
                       const float* X, const float* W, const float* b,
                       float* Y, void* saved, void* workspace,
                       size_t workspace_bytes, hipStream_t stream);
gnn_status gnn_gcn_bwd(const gnn_csr* csr, const gnn_layer* layer,
                       const float* X, const float* W, const float* Y,
                       const float* dY, const void* saved, float* dX,
                       float* dW, float* db, void* workspace,
                       size_t workspace_bytes, hipStream_t stream);

/* MixHop (Eq. "mixhop forward"), K >= 0 hops:
 *   Y = ReLU( X W_0 || A_hat X W_1 || ... || A_hat^K X W_K  + b )
 * Y is n x (K+1)h (stride ld_y >= (K+1)h), hop k in columns [kh, (k+1)h);
 * W is f_in x (K+1)h row-major with W_k in the same columns; b is [(K+1)h]
 * or NULL.  The features are propagated first (A_hat^k X for k = 1..K, kept
 * in `saved`); layer->order must be 0 or 1.  Backward: G = dY * 1[Y > 0],
 * G_k its hop-k columns; dW_k = (A_hat^k X)^T G_k (dW laid out like W);
 * dX = sum_k (A_hat^k)^T G_k W_k^T (may be NULL); db = column sums of G
 * (may be NULL). */
size_t gnn_mixhop_saved_bytes(const gnn_csr* csr, const gnn_layer* layer,
                              int32_t K);
size_t gnn_mixhop_workspace_bytes(const gnn_csr* csr, const gnn_layer* layer,
                                  int32_t K);
gnn_status gnn_mixhop_fwd(const gnn_csr* csr, const gnn_layer* layer,
                          int32_t K, const float* X, const float* W,
                          const float* b, float* Y, void* saved,
                          void* workspace, size_t workspace_bytes,
                          hipStream_t stream);
gnn_status gnn_mixhop_bwd(const gnn_csr* csr, const gnn_layer* layer,
                          int32_t K, const float* X, const float* W,
                          const float* Y, const float* dY, const void* saved,
                          float* dX, float* dW, float* db, void* workspace,
                          size_t workspace_bytes, hipStream_t stream);

/* ----------------------------------------------------------- GAT layer */

/* Section 2.1, Eqs. "gat forward" and "gat attention": on the stored
 * entries (u, v) of the subgraph (edges and self loops; the CSR's values
 * are not used, its pattern must be symmetric and its plan built),
 *   P = X W,  att_uv = LeakyReLU(a1 . P_u + a2 . P_v)  (slope alpha in
 *   [0, 1] below 0),  Y = ReLU(A_att P)
 * with a = [a1; a2] (2h floats, device).  layer: f_in, h, ld_x, ld_y
 * (Y is n x h), ld_dx; order is ignored; flags: GNN_FLAG_BF16 or
 * GNN_FLAG_F32_MFMA for the products.  att_out (nnz floats, may be NULL) receives the attention
 * values in CSR order.  `saved` (gnn_gat_saved_bytes) carries P, the
 * scores and the attention values from the forward to the backward call.
 * Backward: dW (f_in x h), da (2h) and optionally dX, by the chain rule
 * (the per-entry products G_u . P_v form an SDDMM).  No output may overlap
 * an input, another output or the workspace (gnn_gat_workspace_bytes). */
size_t gnn_gat_saved_bytes(const gnn_csr* csr, const gnn_layer* layer);
size_t gnn_gat_workspace_bytes(const gnn_csr* csr, const gnn_layer* layer);
gnn_status gnn_gat_fwd(const gnn_csr* csr, const gnn_layer* layer, const float* X,
                       const float* W, const float* a, float alpha, float* Y,
                       float* att_out, void* saved, void* workspace,
                       size_t workspace_bytes, hipStream_t stream);
gnn_status gnn_gat_bwd(const gnn_csr* csr, const gnn_layer* layer, const float* X,
                       const float* W, const float* a, float alpha, const float* Y,
                       const float* dY, const void* saved, float* dX, float* dW,
                       float* da, void* workspace, size_t workspace_bytes,
                       hipStream_t stream);

/* --------------------------------------- classifier, loss, weight update */

/* Section 3.1 (Eqs. "mlp forward", "loss forward") and Algorithm 1: the
 * classifier head and loss that follow the GNN layers, with the gradients
 * of Section 5.1:
 *   XM = ReLU(X W)      X n x f (stride ld_x), W f x C row-major
 *   Y  = row softmax of XM (GNN_LOSS_SOFTMAX) or sigmoid(XM) element-wise
 *        (GNN_LOSS_SIGMOID)
 *   loss = (1/n) sum over rows of the cross-entropy of Y against T
 *        (n x C, stride ld_t, entries 0 or 1; one 1 per row for softmax)
 *   G  = (Y - T) / n * 1[XM > 0];   dW = X^T G (f x C);   dX = G W^T
 * `loss` is one float of device memory.  Optional outputs (NULL to skip):
 * xm = X_MLP (n x C, stride ld_xm), probs = Y (stride ld_p), dX (stride
 * ld_dx).  flags: GNN_FLAG_BF16 or GNN_FLAG_F32_MFMA for the three products.  The loss is summed
 * in a fixed order (bit-reproducible).  No output may overlap an input,
 * another output or the workspace.  Workspace:
 * gnn_classifier_workspace_bytes(n, f, C).  n = 0 gives loss 0 and dW = 0. */
#define GNN_LOSS_SOFTMAX 0
#define GNN_LOSS_SIGMOID 1
size_t gnn_classifier_workspace_bytes(int32_t n, int32_t f, int32_t C);
gnn_status gnn_classifier(int32_t n, int32_t f, int32_t C, int32_t kind,
                          uint32_t flags, const float* X, int64_t ld_x,
                          const float* W, const float* T, int64_t ld_t,
                          float* xm, int64_t ld_xm, float* probs, int64_t ld_p,
                          float* loss, float* dW, float* dX, int64_t ld_dx,
                          void* workspace, size_t workspace_bytes,
                          hipStream_t stream);

/* Weight update of Algorithm 1 (which leaves the rule open: plain gradient
 * descent, or Adam) on `count` contiguous floats (device):
 *   SGD:   W -= lr G
 *   Adam:  m = b1 m + (1 - b1) G;  v = b2 v + (1 - b2) G^2;
 *          W -= lr (m / (1 - b1^t)) / (sqrt(v / (1 - b2^t)) + eps),  t >= 1
 * m and v (zero before the first step) are updated in place; no two
 * arrays may overlap.  The hyperparameters are host doubles: 1 - b1,
 * 1 - b2 and the bias corrections are formed in double and rounded once to
 * fp32, the precision of the update itself. */
gnn_status gnn_sgd_step(int64_t count, float* W, const float* G, double lr,
                        hipStream_t stream);
gnn_status gnn_adam_step(int64_t count, float* W, const float* G, float* m,
                         float* v, double lr, double beta1, double beta2,
                         double eps, int32_t t, hipStream_t stream);

/* ------------------------------------------- subgraph preparation (prep) */

/* The subgraph of the full training graph induced by a sampled node set
 * (the last step of the samplers, Section 4, Algorithms 2 and 3; Algorithm
 * 1's adjacency matrix of G_s), on the GPU against a full graph resident in
 * device memory:
 *   full graph: n_full nodes, CSR with int64 row pointers indptr (n_full + 1)
 *     and int32 indices (nnz_full), rows sorted, symmetric, unweighted;
 *   nodes: n_s full-graph ids (device), strictly ascending; node nodes[i]
 *     becomes node i of the subgraph;
 *   result: CSR sub_indptr (n_s + 1), sub_indices / sub_values (room for
 *     `capacity` entries; the sum over V_s of (full degree + 1) always
 *     suffices), every node with its self loop, rows sorted; values
 *     1/len_u (GNN_NORM_ROW: D^-1 A of Eq. "graphsage forward", D counting
 *     the stored entries) or 1/sqrt(len_u len_v) (GNN_NORM_SYM, the GCN
 *     layer's normalisation of Section 2.1);
 *   nnz_out (device int64) receives the number of stored entries;
 *   status_out (device int32) receives 0, or bits 1 (an id out of range:
 *     that row keeps its self loop only), 2 (ids not strictly ascending:
 *     the result is not meaningful), 4 (more entries than capacity: the
 *     excess is not written);
 *   map: n_full int32 of device scratch, all -1 on entry, all -1 again
 *     when the call's work completes (it maps full ids to V_s positions).
 * Nothing is read back to the host: the caller copies nnz_out / status_out
 * when it needs them.  Workspace: gnn_induce_workspace_bytes(n_s). */
#define GNN_NORM_ROW 0
#define GNN_NORM_SYM 1
size_t gnn_induce_workspace_bytes(int32_t n_s);
gnn_status gnn_induce_subgraph(int64_t n_full, int64_t nnz_full,
                               const int64_t* indptr, const int32_t* indices,
                               int32_t n_s, const int32_t* nodes, int32_t norm,
                               int32_t* map, int64_t capacity,
                               int32_t* sub_indptr, int32_t* sub_indices,
                               float* sub_values, int64_t* nnz_out,
                               int32_t* status_out, void* workspace,
                               size_t workspace_bytes, hipStream_t stream);

/* Algorithm 1's lookup of the minibatch features / labels by V_s:
 * dst row r = src row index[r] (width floats; src has src_rows rows of
 * stride ld_src, dst stride ld_dst); an index outside [0, src_rows) gives a
 * row of zeros.  dst may not overlap src or index. */
gnn_status gnn_gather_rows(int32_t rows, const int32_t* index, int32_t width,
                           const float* src, int64_t ld_src, int64_t src_rows,
                           float* dst, int64_t ld_dst, hipStream_t stream);

/* ------------------------------------------ sampling and the pool (host) */

/* Frontier sampling (Section 4.1, Algorithm 2) through the Dashboard of
 * Section 4.2 (Algorithms 3 and 4), host code.  Full graph in HOST memory
 * (int64 indptr of n_full + 1, int32 indices, symmetric, rows sorted).
 * m: frontier size; budget: n of Algorithm 2 (budget - m frontier updates;
 * budget >= m); eta >= 1: Dashboard enlargement (eta * m * d slots, d the
 * mean degree); clip > 1 drops |V_s| mod clip nodes chosen uniformly (the
 * node clipping of Section 6.2; 0 or 1: none).  V_s is the initial frontier
 * plus every node that enters the frontier, returned sorted and distinct in
 * `nodes` (room for `budget` ints), its size in *n_nodes.  The result is a
 * function of (graph, parameters, seed, id) only; random numbers are
 * SplitMix64 outputs used as a counter-based generator (stream start
 * states: outputs 4 id + k of the generator started at seed; k = 0 initial
 * frontier, 1 probes, 2 neighbour choice, 3 clipping; an integer below K is
 * floor(r K / 2^64)). */
gnn_status gnn_frontier_sample(int64_t n_full, const int64_t* indptr,
                               const int32_t* indices, int32_t m, int32_t budget,
                               double eta, int32_t clip, uint64_t seed, int64_t id,
                               int32_t* nodes, int32_t* n_nodes);

/* The subgraph pool of Algorithm 8: `threads` worker threads sample
 * subgraphs id = 0, 1, 2, ... (each exactly as gnn_frontier_sample with
 * that id) and keep at most `depth` of them ready; gnn_sampler_next hands
 * them out in id order, blocking until the next one is ready.  The graph
 * arrays must stay valid and unchanged until gnn_sampler_destroy, which
 * stops and joins the workers.  One consumer thread per pool. */
typedef struct gnn_sampler gnn_sampler;
gnn_status gnn_sampler_create(int64_t n_full, const int64_t* indptr,
                              const int32_t* indices, int32_t m, int32_t budget,
                              double eta, int32_t clip, uint64_t seed,
                              int32_t threads, int32_t depth, gnn_sampler** out);
gnn_status gnn_sampler_next(gnn_sampler* s, int32_t* nodes, int32_t* n_nodes,
                            int64_t* id);
void gnn_sampler_destroy(gnn_sampler* s);

/* ------------------------------------------------------------- kernels */

/* Feature / gradient propagation alone (Section 5.1's first kernel, the
 * per-slice product of Section 5.3, Algorithm 7):
 *   out = A_s . in        (transpose = 0, uses csr->values)
 *   out = (A_s)^T . in    (transpose = 1, uses csr->values_t)
 * in and out are n x w with strides ld_in, ld_out; needs csr->plan;
 * `workspace` of gnn_spmm_workspace_bytes(csr, w) bytes (may be NULL if 0;
 * the current kernel needs none and returns 0).  out must not overlap in. */
size_t gnn_spmm_workspace_bytes(const gnn_csr* csr, int32_t w);
gnn_status gnn_spmm(const gnn_csr* csr, int32_t transpose, int32_t w,
                    const float* in, int64_t ld_in, float* out,
                    int64_t ld_out, void* workspace, size_t workspace_bytes,
                    hipStream_t stream);

/* Measurement aid, not part of the method: the gathers of gnn_spmm alone.
 * It runs gnn_spmm's grid, column slices, lane groups, entry order and
 * loads (index, value, neighbour row slice) but keeps one sum per lane for
 * all of its entries instead of one per row: no per-entry row reads, no row
 * closing, no finishing of rows shared between lane groups.  Each plan
 * window's column totals (in a fixed order) go to the window's first row,
 * zeros to its other rows, so every row of `out` is written once and the
 * column sums of `out` equal those of A_s . in (resp. (A_s)^T . in).  Its
 * time bounds from below what the aggregation's gather order costs on the
 * device.  Same arguments and checks as gnn_spmm (no workspace); rows of
 * `in` and `out` must start 16-byte aligned (else GNN_ERR_UNSUPPORTED). */
gnn_status gnn_spmm_gather_floor(const gnn_csr* csr, int32_t transpose,
                                 int32_t w, const float* in, int64_t ld_in,
                                 float* out, int64_t ld_out, hipStream_t stream);

/* Dense weight transformation alone (Section 5.1's second kernel):
 *   C = op(A) op(B),  C is M x N (stride ldc),
 *   op(A) = A (M x K, stride lda)  or A^T with A stored K x M (trans_a = 1),
 *   op(B) = B (K x N, stride ldb)  or B^T with B stored N x K (trans_b = 1).
 * flags: GNN_FLAG_BF16 or GNN_FLAG_F32_MFMA (neither: split products).
 * `workspace` of gnn_gemm_workspace_bytes bytes. */
size_t gnn_gemm_workspace_bytes(int32_t M, int32_t N, int32_t K);
gnn_status gnn_gemm(int32_t trans_a, int32_t trans_b, int32_t M, int32_t N,
                    int32_t K, const float* A, int64_t lda, const float* B,
                    int64_t ldb, float* C, int64_t ldc, uint32_t flags,
                    void* workspace, size_t workspace_bytes,
                    hipStream_t stream);

/* Measurement aid, not part of the method: the sustained rate of the
 * device's matrix cores, against which the products' rates are read.
 * Launches `blocks` workgroups of 512 threads (eight wavefronts, two
 * workgroups per CU as in the split-product GEMM); every wavefront issues
 * 4 x `iters` MFMAs on register operands into four independent accumulators,
 * with no memory traffic in the loop:
 *   GNN_PROBE_MFMA_BF16  v_mfma_f32_32x32x16_bf16, 32768 flop each
 *   GNN_PROBE_MFMA_F32   v_mfma_f32_32x32x2_f32,    4096 flop each
 * so one launch does blocks x 8 x 4 x iters x (flop each).  The caller times
 * the launch (events on `stream`) for the rate.  `sink` (device, blocks x
 * 512 floats, 4-byte aligned) receives each thread's accumulator sum.
 * `clocks` (device, two 8-byte-aligned uint64) receives the shader-clock
 * cycles (s_memtime) and the 100 MHz real-time ticks (s_memrealtime) that
 * the first wavefront of workgroup 0 counted over its loop: cycles / ticks
 * x 0.1 is the shader clock in GHz under this load.  Errors: an unknown
 * kind GNN_ERR_UNSUPPORTED, blocks or iters outside [1, max]
 * GNN_ERR_SHAPE, a NULL pointer GNN_ERR_NULL, misaligned pointers
 * GNN_ERR_UNSUPPORTED, `sink` overlapping `clocks` GNN_ERR_ALIAS. */
#define GNN_PROBE_MFMA_BF16 0
#define GNN_PROBE_MFMA_F32 1
#define GNN_PROBE_MAX_BLOCKS 65536
#define GNN_PROBE_MAX_ITERS 100000
gnn_status gnn_mfma_rate_probe(int32_t kind, int32_t blocks, int32_t iters,
                               float* sink, uint64_t* clocks, hipStream_t stream);

/* ----------------------------------------------------- kernel timing */

/* Kernels timed by the optional event timer. */
#define GNN_K_SPMM 0          /* aggregation (one kernel per product) */
#define GNN_K_SPMM_REDUCE 1   /* reserved: no separate reduction is launched */
#define GNN_K_GEMM_NN 2       /* C = A B            (forward transforms) */
#define GNN_K_GEMM_TN 3       /* C = A^T B          (weight gradients) */
#define GNN_K_GEMM_NT 4       /* C = A B^T          (input gradients) */
#define GNN_K_GEMM_TT 5       /* C = A^T B^T */
#define GNN_K_GEMM_REDUCE 6   /* split-K partial reduction */
#define GNN_K_MASK 7          /* ReLU mask of the output gradient */
#define GNN_K_COLSUM 8        /* bias-gradient column sums */
#define GNN_K_PLAN 9          /* aggregation plan build */
#define GNN_K_TRANSPOSE 10    /* transposed values (Algorithm 6) */
#define GNN_K_LOSS 11         /* classifier loss and its gradient */
#define GNN_K_UPDATE 12       /* weight update (SGD or Adam) */
#define GNN_K_INDUCE 13       /* induced subgraph on the GPU */
#define GNN_K_GATHER 14       /* feature / label row gather */
#define GNN_K_SDDMM 15        /* GAT per-entry dot products */
#define GNN_K_WSPLIT 16       /* weights split into bf16 pieces (split products) */
#define GNN_K_COUNT 17

/* When enabled, every kernel launch is bracketed by a pair of HIP events on
 * its stream.  gnn_timer_read synchronises on the recorded events and
 * returns, for one kernel id since the last reset, the summed milliseconds,
 * the launch count and the summed algorithmic work of those launches:
 * bytes for memory-bound kernels (aggregation: 4(n+1) + 8 nnz + 8 n w per
 * call, counted on GNN_K_SPMM), flops for the GEMMs (2 M N K).  Host-side
 * bookkeeping only; not thread safe. */
gnn_status gnn_timer_enable(int32_t enable);
gnn_status gnn_timer_reset(void);
gnn_status gnn_timer_read(int32_t kernel, double* ms, int64_t* launches,
                          double* work);

#ifdef __cplusplus
}
#endif
#endif /* GNNPROP_H */
