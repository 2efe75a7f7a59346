/*
 * CPU oracle for one GNN layer's feature propagation (GraphSAGE, and the
 * GCN and MixHop variants), forward and backward, on a sampled subgraph
 * ("Accurate, Efficient and Scalable Training of Graph Neural Networks",
 * Zeng et al.).
 *
 * TEST INFRASTRUCTURE ONLY.  This library is the slow, obviously-correct
 * reference that the GPU path is checked against.  Only the test suite, the
 * smoke check and the benchmark's CPU-baseline leg may load it.  It shares no
 * source, header, table or helper with the GPU library.
 *
 * Conventions
 *   - every floating-point input and output is double (the paper trains in
 *     double precision, Section 5.3 footnote); all sums accumulate in double
 *     in a fixed order, so results do not depend on the thread count;
 *   - dense matrices are row-major and contiguous (leading dimension = width);
 *   - the subgraph adjacency is CSR: indptr[n+1], indices[nnz] (column ids,
 *     ascending within a row), values[nnz];
 *   - a layer's output is [self half | neighbour half], each h wide.
 */
#ifndef GNN_ORACLE_H
#define GNN_ORACLE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Section 2.1, Eq. "graphsage forward": out = A_s . in  (CSR order sum). */
void oracle_spmm(int32_t n, const int32_t* indptr, const int32_t* indices,
                 const double* values, int32_t w, const double* in,
                 double* out);

/* out = (A_s)^T . in, applied as a scatter over the CSR of A_s:
 * out[u,:] = sum over stored (v,u) of A_s[v,u] * in[v,:], v ascending.
 * Independent of Algorithm 6 and of any symmetry of the pattern. */
void oracle_spmm_transpose(int32_t n, const int32_t* indptr,
                           const int32_t* indices, const double* values,
                           int32_t w, const double* in, double* out);

/* Section 5.2: values of (A_s)^T on the same indptr/indices (the array
 * Algorithm 6 builds), written from its definition: entry (u,v) takes the
 * value stored at (v,u).  Requires a symmetric pattern.  Returns 0, or -1
 * if some (v,u) has no stored (u,v) counterpart. */
int32_t oracle_transpose_values(int32_t n, const int32_t* indptr,
                                const int32_t* indices, const double* values,
                                double* values_t);

/* Section 6.1: computation order of A.W1.W2 (A n-by-n sparse, W1 n-by-f1,
 * W2 f1-by-f2).  Returns 1 for (A W1) W2, 2 for A (W1 W2). */
int32_t oracle_choose_order(int64_t f1, int64_t f2);

/* Dense products, ascending-k sums.  C is M x N.
 *   nn: C = A B      A: M x K, B: K x N
 *   tn: C = A^T B    A: K x M, B: K x N
 *   nt: C = A B^T    A: M x K, B: N x K                                    */
void oracle_mm_nn(int32_t M, int32_t N, int32_t K, const double* A,
                  const double* B, double* C);
void oracle_mm_tn(int32_t M, int32_t N, int32_t K, const double* A,
                  const double* B, double* C);
void oracle_mm_nt(int32_t M, int32_t N, int32_t K, const double* A,
                  const double* B, double* C);

/* Forward of one layer (Eq. "graphsage forward", self half first):
 *   S = A_s X                                  (n x f_in, may be NULL)
 *   Y = ReLU([X W_self + b_self || S W_neigh + b_neigh])   (n x 2h)
 * b_self / b_neigh may be NULL (no bias, the paper's form). */
void oracle_sage_fwd(int32_t n, const int32_t* indptr, const int32_t* indices,
                     const double* values, int32_t f_in, int32_t h,
                     const double* X, const double* W_self,
                     const double* W_neigh, const double* b_self,
                     const double* b_neigh, double* Y, double* S);

/* Backward of one layer (Section 5.1, Eq. "gcn backward"), given the
 * layer output Y (its sign pattern is the ReLU mask) and dY = dL/dY:
 *   G       = dY * 1[Y > 0]            G_s = G[:, :h], G_n = G[:, h:]
 *   dW_self = X^T G_s
 *   dW_neigh= (A_s X)^T G_n
 *   dX      = G_s W_self^T + ((A_s)^T G_n) W_neigh^T
 *   db_*    = column sums of G_*  (db pointers may be NULL)
 * dX may be NULL (skipped). */
void oracle_sage_bwd(int32_t n, const int32_t* indptr, const int32_t* indices,
                     const double* values, int32_t f_in, int32_t h,
                     const double* X, const double* W_self,
                     const double* W_neigh, const double* Y, const double* dY,
                     double* dX, double* dW_self, double* dW_neigh,
                     double* db_self, double* db_neigh);

/* The same definitions evaluated one output at a time, for spot checks of
 * large cases.  rows[] lists node ids; outputs are packed per listed row. */
void oracle_sage_fwd_rows(int32_t n, const int32_t* indptr,
                          const int32_t* indices, const double* values,
                          int32_t f_in, int32_t h, const double* X,
                          const double* W_self, const double* W_neigh,
                          const double* b_self, const double* b_neigh,
                          int32_t nrows, const int32_t* rows, double* Y_rows);

void oracle_sage_bwd_dx_rows(int32_t n, const int32_t* indptr,
                             const int32_t* indices, const double* values,
                             int32_t f_in, int32_t h, const double* W_self,
                             const double* W_neigh, const double* Y,
                             const double* dY, int32_t nrows,
                             const int32_t* rows, double* dX_rows);

/* Entries (ei[k], ej[k]) of dW_self and dW_neigh. */
void oracle_sage_bwd_dw_entries(int32_t n, const int32_t* indptr,
                                const int32_t* indices, const double* values,
                                int32_t f_in, int32_t h, const double* X,
                                const double* Y, const double* dY,
                                int32_t nent, const int32_t* ei,
                                const int32_t* ej, double* dWs_ent,
                                double* dWn_ent);

/* GCN layer (Section 2.1, Eq. "gcn forward"), values = A_hat:
 *   Y = ReLU(A_hat X W + b)                    (n x h; S = A_hat X, may be NULL)
 * Backward (Section 5.1 with only the A_hat terms kept):
 *   G = dY * 1[Y > 0];  dW = (A_hat X)^T G;  dX = A_hat^T G W^T;  db = colsum G */
void oracle_gcn_fwd(int32_t n, const int32_t* indptr, const int32_t* indices,
                    const double* values, int32_t f_in, int32_t h,
                    const double* X, const double* W, const double* b,
                    double* Y, double* S);
void oracle_gcn_bwd(int32_t n, const int32_t* indptr, const int32_t* indices,
                    const double* values, int32_t f_in, int32_t h,
                    const double* X, const double* W, const double* Y,
                    const double* dY, double* dX, double* dW, double* db);

/* MixHop layer (Section 2.1, Eq. "mixhop forward"), values = A_hat:
 *   Y = ReLU( X W_0 || A_hat X W_1 || ... || A_hat^K X W_K  + b )
 * Y is n x (K+1)h, W is f_in x (K+1)h (W_k in columns [kh, (k+1)h)), b is
 * (K+1)h (may be NULL).  Backward: G = dY * 1[Y > 0], G_k its hop-k columns;
 *   dW_k = (A_hat^k X)^T G_k;  dX = sum_k (A_hat^k)^T G_k W_k^T;  db = colsum G */
void oracle_mixhop_fwd(int32_t n, const int32_t* indptr,
                       const int32_t* indices, const double* values,
                       int32_t K, int32_t f_in, int32_t h, const double* X,
                       const double* W, const double* b, double* Y);
void oracle_mixhop_bwd(int32_t n, const int32_t* indptr,
                       const int32_t* indices, const double* values,
                       int32_t K, int32_t f_in, int32_t h, const double* X,
                       const double* W, const double* Y, const double* dY,
                       double* dX, double* dW, double* db);

/* Classifier head and loss (Section 3.1, Algorithm 1): Z = X W (n x C),
 * X_MLP = ReLU(Z), Y = sigma(X_MLP) with sigma a row softmax (kind 0) or an
 * element-wise sigmoid (kind 1); L = mean over rows of the cross-entropy
 * against T (n x C, 0/1).  Gradients (Section 5.1): dL/dX_MLP = (Y - T)/n,
 * G = that * 1[X_MLP > 0], dW = X^T G, dX = G W^T.  probs (Y) and dX may be
 * NULL.  Returns L.  relu_on (n x C bytes, may be NULL) gives the MLP ReLU's
 * decision instead of Z > 0. */
double oracle_classifier(int32_t n, int32_t f, int32_t C, const double* X,
                         const double* W, const double* T, int32_t kind,
                         double* probs, double* dW, double* dX,
                         const uint8_t* relu_on);

/* Weight updates: plain gradient step, and Adam with bias correction at
 * step t >= 1 (moments m, v updated in place). */
void oracle_sgd(int64_t count, double* W, const double* g, double lr);
void oracle_adam(int64_t count, double* W, const double* g, double* m,
                 double* v, double lr, double b1, double b2, double eps,
                 int32_t t);

/* bfloat16 rounding of GEMM operands for the reduced-precision mode: each
 * value is first taken as float (the storage format), then rounded to the
 * nearest bfloat16 (8 significant bits), ties to even; NaN stays NaN. */
void oracle_round_bf16(int64_t count, const double* in, double* out);

/* Number of OpenMP threads the oracle runs with. */
int32_t oracle_num_threads(void);
void oracle_set_num_threads(int32_t n);

/* Induced subgraph of a full graph (int64 row pointers) on the sorted,
 * distinct node list `nodes` (node nodes[i] becomes i), self loops added,
 * values 1/len_u (norm 0) or 1/sqrt(len_u len_v) (norm 1).  Returns nnz. */
int64_t oracle_induce(int64_t n_full, const int64_t* indptr,
                      const int32_t* indices, int32_t n_s,
                      const int32_t* nodes, int32_t norm, int32_t* out_indptr,
                      int32_t* out_indices, double* out_values);

/* GAT layer (Section 2.1): P = X W, att_uv = LeakyReLU(a1 . P_u + a2 . P_v)
 * on the stored entries (slope alpha below 0), Y = ReLU(A_att P); att
 * (nnz) may be NULL.  Backward by the chain rule; dX may be NULL; da has
 * 2h entries; z_pos (nnz bytes, may be NULL) gives the LeakyReLU's
 * decisions. */
void oracle_gat_fwd(int32_t n, const int32_t* indptr, const int32_t* indices,
                    int32_t f_in, int32_t h, const double* X, const double* W,
                    const double* a, double alpha, double* Y, double* att);
void oracle_gat_bwd(int32_t n, const int32_t* indptr, const int32_t* indices,
                    int32_t f_in, int32_t h, const double* X, const double* W,
                    const double* a, double alpha, const double* Y,
                    const double* dY, double* dX, double* dW, double* da,
                    const uint8_t* z_pos);

#ifdef __cplusplus
}
#endif
#endif
