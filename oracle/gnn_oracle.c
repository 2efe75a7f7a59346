/*
 * CPU oracle for GraphSAGE feature propagation on a sampled subgraph.
 * TEST INFRASTRUCTURE ONLY -- see gnn_oracle.h.  Plain loops, double
 * precision throughout, fixed summation order, OpenMP only over independent
 * outputs.  Shares nothing with the GPU library.
 */
#include "gnn_oracle.h"

#include <math.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

int32_t oracle_num_threads(void) {
#ifdef _OPENMP
  return (int32_t)omp_get_max_threads();
#else
  return 1;
#endif
}

/* Threads of the following parallel regions (results do not depend on it). */
void oracle_set_num_threads(int32_t n) {
#ifdef _OPENMP
  if (n > 0) omp_set_num_threads(n);
#else
  (void)n;
#endif
}

/* bfloat16 keeps the sign, the 8 exponent bits and the top 7 fraction bits
 * of a float.  Rounding to nearest, ties to even, adds 0x7fff plus the
 * lowest kept bit to the 32-bit pattern and truncates the low 16 bits. */
void oracle_round_bf16(int64_t count, const double* in, double* out) {
  for (int64_t i = 0; i < count; ++i) {
    float f = (float)in[i];
    uint32_t u;
    memcpy(&u, &f, sizeof u);
    if (f != f) {
      out[i] = in[i];
      continue;
    }
    u = (u + 0x7fffu + ((u >> 16) & 1u)) & 0xffff0000u;
    memcpy(&f, &u, sizeof f);
    out[i] = (double)f;
  }
}

/* ------------------------------------------------------------------ SpMM */

/* Feature aggregation A_s . X (Section 2.1; Section 5.3 for the operation
 * itself): row v of the output is the values-weighted sum of the input rows
 * of v's neighbours, taken in CSR order. */
void oracle_spmm(int32_t n, const int32_t* indptr, const int32_t* indices,
                 const double* values, int32_t w, const double* in,
                 double* out) {
#pragma omp parallel for schedule(dynamic, 16)
  for (int32_t v = 0; v < n; ++v) {
    double* o = out + (int64_t)v * w;
    for (int32_t c = 0; c < w; ++c) o[c] = 0.0;
    for (int32_t j = indptr[v]; j < indptr[v + 1]; ++j) {
      const double a = values[j];
      const double* x = in + (int64_t)indices[j] * w;
      for (int32_t c = 0; c < w; ++c) o[c] += a * x[c];
    }
  }
}

/* Transposed aggregation (A_s)^T . in used by the input gradient (Section
 * 5.1).  Entry (v,u) of A_s is entry (u,v) of the transpose, so every stored
 * (v,u) adds A_s[v,u] * in[v,:] into out[u,:].  Each thread owns a range of
 * feature columns (all rows), so every output element is summed by one
 * thread in ascending v. */
void oracle_spmm_transpose(int32_t n, const int32_t* indptr,
                           const int32_t* indices, const double* values,
                           int32_t w, const double* in, double* out) {
  memset(out, 0, sizeof(double) * (size_t)n * (size_t)w);
#pragma omp parallel
  {
    int nt = 1, t = 0;
#ifdef _OPENMP
    nt = omp_get_num_threads();
    t = omp_get_thread_num();
#endif
    const int32_t c0 = (int32_t)((int64_t)w * t / nt);
    const int32_t c1 = (int32_t)((int64_t)w * (t + 1) / nt);
    for (int32_t v = 0; v < n; ++v) {
      const double* x = in + (int64_t)v * w;
      for (int32_t j = indptr[v]; j < indptr[v + 1]; ++j) {
        const double a = values[j];
        double* o = out + (int64_t)indices[j] * w;
        for (int32_t c = c0; c < c1; ++c) o[c] += a * x[c];
      }
    }
  }
}

/* Transposed values on the pattern of A_s (Section 5.2): the transpose
 * holds A_s[v,u] at position (u,v), so each stored entry k = (u,v) of row u
 * takes the value stored at (v,u), which a plain scan of row v finds.  This
 * is the defining property itself; Algorithm 6 produces the same array in
 * one pass.  Returns -1 if some (v,u) is not stored (the pattern is not
 * symmetric and the transpose does not fit it). */
int32_t oracle_transpose_values(int32_t n, const int32_t* indptr,
                                const int32_t* indices, const double* values,
                                double* values_t) {
  int32_t status = 0;
#pragma omp parallel for schedule(dynamic, 64) reduction(min : status)
  for (int32_t u = 0; u < n; ++u) {
    for (int32_t k = indptr[u]; k < indptr[u + 1]; ++k) {
      const int32_t v = indices[k];
      int32_t at = -1;
      for (int32_t j = indptr[v]; j < indptr[v + 1]; ++j)
        if (indices[j] == u) {
          at = j;
          break;
        }
      if (at < 0) {
        status = -1;
        continue;
      }
      values_t[k] = values[at];
    }
  }
  return status;
}

/* Section 6.1: order 1 costs delta n^2 f1 + n f1 f2 MACs, order 2 costs
 * delta n^2 f2 + n f1 f2; the shared term cancels, so order 1 wins when
 * f1 < f2.  A tie costs the same either way and is given to order 1. */
int32_t oracle_choose_order(int64_t f1, int64_t f2) {
  return f1 <= f2 ? 1 : 2;
}

/* ---------------------------------------------------------- dense products */

void oracle_mm_nn(int32_t M, int32_t N, int32_t K, const double* A,
                  const double* B, double* C) {
#pragma omp parallel for schedule(static)
  for (int32_t i = 0; i < M; ++i) {
    double* c = C + (int64_t)i * N;
    for (int32_t j = 0; j < N; ++j) c[j] = 0.0;
    for (int32_t k = 0; k < K; ++k) {
      const double a = A[(int64_t)i * K + k];
      const double* b = B + (int64_t)k * N;
      for (int32_t j = 0; j < N; ++j) c[j] += a * b[j];
    }
  }
}

void oracle_mm_tn(int32_t M, int32_t N, int32_t K, const double* A,
                  const double* B, double* C) {
#pragma omp parallel for schedule(static)
  for (int32_t i = 0; i < M; ++i) {
    double* c = C + (int64_t)i * N;
    for (int32_t j = 0; j < N; ++j) c[j] = 0.0;
    for (int32_t k = 0; k < K; ++k) {
      const double a = A[(int64_t)k * M + i];
      const double* b = B + (int64_t)k * N;
      for (int32_t j = 0; j < N; ++j) c[j] += a * b[j];
    }
  }
}

void oracle_mm_nt(int32_t M, int32_t N, int32_t K, const double* A,
                  const double* B, double* C) {
#pragma omp parallel for schedule(static)
  for (int32_t i = 0; i < M; ++i) {
    const double* a = A + (int64_t)i * K;
    for (int32_t j = 0; j < N; ++j) {
      const double* b = B + (int64_t)j * K;
      double s = 0.0;
      for (int32_t k = 0; k < K; ++k) s += a[k] * b[k];
      C[(int64_t)i * N + j] = s;
    }
  }
}

/* ------------------------------------------------------------- one layer */

static double relu(double z) { return z > 0.0 ? z : 0.0; }

/* Eq. "graphsage forward": X_out = ReLU( X W_self || (A_s X) W_neigh ),
 * with the self half in columns [0,h) (the column split the gradient
 * equations of Section 5.1 use) and an optional per-half bias added
 * before the activation. */
void oracle_sage_fwd(int32_t n, const int32_t* indptr, const int32_t* indices,
                     const double* values, int32_t f_in, int32_t h,
                     const double* X, const double* W_self,
                     const double* W_neigh, const double* b_self,
                     const double* b_neigh, double* Y, double* S_out) {
  const size_t nf = (size_t)n * (size_t)f_in, nh = (size_t)n * (size_t)h;
  double* S = S_out ? S_out : (double*)malloc(sizeof(double) * (nf ? nf : 1));
  double* Zs = (double*)malloc(sizeof(double) * (nh ? nh : 1));
  double* Zn = (double*)malloc(sizeof(double) * (nh ? nh : 1));
  oracle_spmm(n, indptr, indices, values, f_in, X, S); /* A_s X */
  oracle_mm_nn(n, h, f_in, X, W_self, Zs);              /* X W_self */
  oracle_mm_nn(n, h, f_in, S, W_neigh, Zn);             /* (A_s X) W_neigh */
#pragma omp parallel for schedule(static)
  for (int32_t v = 0; v < n; ++v) {
    double* y = Y + (int64_t)v * 2 * h;
    for (int32_t c = 0; c < h; ++c) {
      const double zs = Zs[(int64_t)v * h + c] + (b_self ? b_self[c] : 0.0);
      const double zn = Zn[(int64_t)v * h + c] + (b_neigh ? b_neigh[c] : 0.0);
      y[c] = relu(zs);
      y[h + c] = relu(zn);
    }
  }
  free(Zs);
  free(Zn);
  if (!S_out) free(S);
}

/* mask(): the derivative of the layer's own ReLU, 1 where the output is
 * positive and 0 elsewhere (0 is taken at the kink). */
static void masked_grad(int32_t n, int32_t h, const double* Y,
                        const double* dY, double* Gs, double* Gn) {
#pragma omp parallel for schedule(static)
  for (int32_t v = 0; v < n; ++v) {
    for (int32_t c = 0; c < h; ++c) {
      const int64_t a = (int64_t)v * 2 * h + c, b = a + h;
      Gs[(int64_t)v * h + c] = Y[a] > 0.0 ? dY[a] : 0.0;
      Gn[(int64_t)v * h + c] = Y[b] > 0.0 ? dY[b] : 0.0;
    }
  }
}

/* Section 5.1, Eq. "gcn backward" (stated there for GraphSAGE). */
void oracle_sage_bwd(int32_t n, const int32_t* indptr, const int32_t* indices,
                     const double* values, int32_t f_in, int32_t h,
                     const double* X, const double* W_self,
                     const double* W_neigh, const double* Y, const double* dY,
                     double* dX, double* dW_self, double* dW_neigh,
                     double* db_self, double* db_neigh) {
  const size_t nf = (size_t)n * (size_t)f_in, nh = (size_t)n * (size_t)h;
  double* Gs = (double*)malloc(sizeof(double) * (nh ? nh : 1));
  double* Gn = (double*)malloc(sizeof(double) * (nh ? nh : 1));
  double* S = (double*)malloc(sizeof(double) * (nf ? nf : 1));
  masked_grad(n, h, Y, dY, Gs, Gn);

  oracle_mm_tn(f_in, h, n, X, Gs, dW_self);            /* X^T G_s */
  oracle_spmm(n, indptr, indices, values, f_in, X, S);  /* A_s X */
  oracle_mm_tn(f_in, h, n, S, Gn, dW_neigh);           /* (A_s X)^T G_n */

  if (db_self || db_neigh) {
    for (int32_t c = 0; c < h; ++c) {
      double ss = 0.0, sn = 0.0;
      for (int32_t v = 0; v < n; ++v) {
        ss += Gs[(int64_t)v * h + c];
        sn += Gn[(int64_t)v * h + c];
      }
      if (db_self) db_self[c] = ss;
      if (db_neigh) db_neigh[c] = sn;
    }
  }

  if (dX) {
    double* T = (double*)malloc(sizeof(double) * (nh ? nh : 1));
    double* R = (double*)malloc(sizeof(double) * (nf ? nf : 1));
    oracle_spmm_transpose(n, indptr, indices, values, h, Gn, T); /* A^T G_n */
    oracle_mm_nt(n, f_in, h, Gs, W_self, dX);                     /* G_s W_s^T */
    oracle_mm_nt(n, f_in, h, T, W_neigh, R);            /* (A^T G_n) W_n^T */
    for (size_t i = 0; i < nf; ++i) dX[i] += R[i];
    free(T);
    free(R);
  }
  free(Gs);
  free(Gn);
  free(S);
}

/* ------------------------------------------------- GCN and MixHop layers */

/* Column sums of an n x w matrix, rows in ascending order. */
static void colsum(int32_t n, int32_t w, const double* G, double* out) {
  for (int32_t c = 0; c < w; ++c) {
    double s = 0.0;
    for (int32_t v = 0; v < n; ++v) s += G[(int64_t)v * w + c];
    out[c] = s;
  }
}

/* G = dY * 1[Y > 0] over an n x w block (the layer's ReLU derivative). */
static void mask_all(int64_t count, const double* Y, const double* dY,
                     double* G) {
  for (int64_t i = 0; i < count; ++i) G[i] = Y[i] > 0.0 ? dY[i] : 0.0;
}

/* Section 2.1, Eq. "gcn forward": Y = ReLU(A_hat X W + b).  values hold
 * A_hat; S (n x f_in, may be NULL) receives A_hat X. */
void oracle_gcn_fwd(int32_t n, const int32_t* indptr, const int32_t* indices,
                    const double* values, int32_t f_in, int32_t h,
                    const double* X, const double* W, const double* b,
                    double* Y, double* S_out) {
  const size_t nf = (size_t)n * (size_t)f_in;
  double* S = S_out ? S_out : (double*)malloc(sizeof(double) * (nf ? nf : 1));
  oracle_spmm(n, indptr, indices, values, f_in, X, S); /* A_hat X */
  oracle_mm_nn(n, h, f_in, S, W, Y);                   /* (A_hat X) W */
  for (int64_t v = 0; v < n; ++v)
    for (int32_t c = 0; c < h; ++c) {
      double* y = Y + v * h + c;
      *y = relu(*y + (b ? b[c] : 0.0));
    }
  if (!S_out) free(S);
}

/* Section 5.1 for GCN: the GraphSAGE gradients with only the A_hat terms
 * kept.  G = dY * 1[Y > 0];  dW = (A_hat X)^T G;  dX = A_hat^T G W^T;
 * db = column sums of G.  dX and db may be NULL. */
void oracle_gcn_bwd(int32_t n, const int32_t* indptr, const int32_t* indices,
                    const double* values, int32_t f_in, int32_t h,
                    const double* X, const double* W, const double* Y,
                    const double* dY, double* dX, double* dW, double* db) {
  const size_t nf = (size_t)n * (size_t)f_in, nh = (size_t)n * (size_t)h;
  double* G = (double*)malloc(sizeof(double) * (nh ? nh : 1));
  double* S = (double*)malloc(sizeof(double) * (nf ? nf : 1));
  mask_all((int64_t)nh, Y, dY, G);
  oracle_spmm(n, indptr, indices, values, f_in, X, S); /* A_hat X */
  oracle_mm_tn(f_in, h, n, S, G, dW);                  /* (A_hat X)^T G */
  if (db) colsum(n, h, G, db);
  if (dX) {
    double* T = (double*)malloc(sizeof(double) * (nh ? nh : 1));
    oracle_spmm_transpose(n, indptr, indices, values, h, G, T); /* A_hat^T G */
    oracle_mm_nt(n, f_in, h, T, W, dX);                         /* (A_hat^T G) W^T */
    free(T);
  }
  free(G);
  free(S);
}

/* Section 2.1, Eq. "mixhop forward": Y = ReLU( ||_{k=0..K} A_hat^k X W_k
 * + b ), Y n x (K+1)h with hop k in columns [k h, (k+1) h).  W is
 * f_in x (K+1)h with W_k in the same columns; A_hat^k X is A_hat applied k
 * times. */
void oracle_mixhop_fwd(int32_t n, const int32_t* indptr,
                       const int32_t* indices, const double* values,
                       int32_t K, int32_t f_in, int32_t h, const double* X,
                       const double* W, const double* b, double* Y) {
  const int32_t wy = (K + 1) * h;
  const size_t nf = (size_t)n * (size_t)f_in, nh = (size_t)n * (size_t)h;
  double* P = (double*)malloc(sizeof(double) * (nf ? nf : 1));  /* A_hat^k X */
  double* Q = (double*)malloc(sizeof(double) * (nf ? nf : 1));
  double* Wk = (double*)malloc(sizeof(double) * ((size_t)f_in * h + 1));
  double* Z = (double*)malloc(sizeof(double) * (nh ? nh : 1));
  memcpy(P, X, sizeof(double) * nf);
  for (int32_t k = 0; k <= K; ++k) {
    if (k > 0) {
      oracle_spmm(n, indptr, indices, values, f_in, P, Q);
      double* s = P;
      P = Q;
      Q = s;
    }
    for (int32_t i = 0; i < f_in; ++i)
      for (int32_t c = 0; c < h; ++c)
        Wk[(int64_t)i * h + c] = W[(int64_t)i * wy + (int64_t)k * h + c];
    oracle_mm_nn(n, h, f_in, P, Wk, Z); /* A_hat^k X W_k */
    for (int64_t v = 0; v < n; ++v)
      for (int32_t c = 0; c < h; ++c)
        Y[v * wy + (int64_t)k * h + c] =
            relu(Z[v * h + c] + (b ? b[(int64_t)k * h + c] : 0.0));
  }
  free(P);
  free(Q);
  free(Wk);
  free(Z);
}

/* Backward for MixHop (Section 5.1 with K paths): G = dY * 1[Y > 0], G_k
 * its hop-k columns;  dW_k = (A_hat^k X)^T G_k;
 * dX = sum_k (A_hat^k)^T G_k W_k^T, each term applying A_hat^T k times to
 * G_k W_k^T;  db = column sums of G.  dX and db may be NULL. */
void oracle_mixhop_bwd(int32_t n, const int32_t* indptr,
                       const int32_t* indices, const double* values,
                       int32_t K, int32_t f_in, int32_t h, const double* X,
                       const double* W, const double* Y, const double* dY,
                       double* dX, double* dW, double* db) {
  const int32_t wy = (K + 1) * h;
  const size_t nf = (size_t)n * (size_t)f_in, nh = (size_t)n * (size_t)h;
  double* G = (double*)malloc(sizeof(double) * ((size_t)n * wy + 1));
  double* Gk = (double*)malloc(sizeof(double) * (nh ? nh : 1));
  double* P = (double*)malloc(sizeof(double) * (nf ? nf : 1));
  double* Q = (double*)malloc(sizeof(double) * (nf ? nf : 1));
  double* Wk = (double*)malloc(sizeof(double) * ((size_t)f_in * h + 1));
  double* D = (double*)malloc(sizeof(double) * ((size_t)f_in * h + 1));
  double* V = (double*)malloc(sizeof(double) * (nf ? nf : 1));
  double* U = (double*)malloc(sizeof(double) * (nf ? nf : 1));
  mask_all((int64_t)n * wy, Y, dY, G);
  if (db) colsum(n, wy, G, db);
  if (dX) memset(dX, 0, sizeof(double) * nf);
  memcpy(P, X, sizeof(double) * nf);
  for (int32_t k = 0; k <= K; ++k) {
    if (k > 0) { /* P = A_hat^k X */
      oracle_spmm(n, indptr, indices, values, f_in, P, Q);
      double* s = P;
      P = Q;
      Q = s;
    }
    for (int64_t v = 0; v < n; ++v)
      for (int32_t c = 0; c < h; ++c)
        Gk[v * h + c] = G[v * wy + (int64_t)k * h + c];
    oracle_mm_tn(f_in, h, n, P, Gk, D); /* (A_hat^k X)^T G_k */
    for (int32_t i = 0; i < f_in; ++i)
      for (int32_t c = 0; c < h; ++c) {
        dW[(int64_t)i * wy + (int64_t)k * h + c] = D[(int64_t)i * h + c];
        Wk[(int64_t)i * h + c] = W[(int64_t)i * wy + (int64_t)k * h + c];
      }
    if (dX) {
      oracle_mm_nt(n, f_in, h, Gk, Wk, V); /* G_k W_k^T */
      for (int32_t j = 0; j < k; ++j) {    /* (A_hat^T)^k applied */
        oracle_spmm_transpose(n, indptr, indices, values, f_in, V, U);
        double* s = V;
        V = U;
        U = s;
      }
      for (size_t i = 0; i < nf; ++i) dX[i] += V[i];
    }
  }
  free(G);
  free(Gk);
  free(P);
  free(Q);
  free(Wk);
  free(D);
  free(V);
  free(U);
}

/* ------------------------------------------------------------- GAT layer */

/* Section 2.1, Eqs. "gat forward" and "gat attention", on the stored
 * entries of the subgraph (its edges and self loops): with P = X W and
 * a = [a1; a2] (2h), entry (u, v) of the attention matrix is
 *   att_uv = LeakyReLU(a1 . P_u + a2 . P_v)   (slope alpha below 0)
 * and Y = ReLU(A_att P).  The CSR's own values are not used.  att (nnz)
 * may be NULL. */
void oracle_gat_fwd(int32_t n, const int32_t* indptr, const int32_t* indices,
                    int32_t f_in, int32_t h, const double* X, const double* W,
                    const double* a, double alpha, double* Y, double* att) {
  const size_t nh = (size_t)n * (size_t)h;
  const int64_t nnz = n > 0 ? indptr[n] : 0;
  double* P = (double*)malloc(sizeof(double) * (nh ? nh : 1));
  double* A = (double*)malloc(sizeof(double) * (nnz ? nnz : 1));
  oracle_mm_nn(n, h, f_in, X, W, P);
  for (int32_t u = 0; u < n; ++u)
    for (int32_t j = indptr[u]; j < indptr[u + 1]; ++j) {
      const int32_t v = indices[j];
      double z = 0.0;
      for (int32_t c = 0; c < h; ++c) z += a[c] * P[(int64_t)u * h + c];
      for (int32_t c = 0; c < h; ++c) z += a[h + c] * P[(int64_t)v * h + c];
      A[j] = z > 0.0 ? z : alpha * z;
    }
  oracle_spmm(n, indptr, indices, A, h, P, Y);
  for (size_t i = 0; i < nh; ++i) Y[i] = relu(Y[i]);
  if (att)
    for (int64_t j = 0; j < nnz; ++j) att[j] = A[j];
  free(A);
  free(P);
}

/* The chain rule through the GAT layer (Section 5.1 does it step by step
 * for the dense parts; the attention's own terms follow from its
 * definition): G = dY * 1[Y > 0]; with Z = A_att P,
 *   dP = A_att^T G  +  sum over entries of dz_uv (a1 at row u, a2 at row v),
 *   dz_uv = (G_u . P_v) * (z_uv > 0 ? 1 : alpha),
 *   da1 = sum dz_uv P_u,  da2 = sum dz_uv P_v,
 *   dW = X^T dP,  dX = dP W^T.
 * dX may be NULL.  z_pos (nnz bytes, may be NULL) supplies the LeakyReLU's
 * decision z_uv > 0 (as another implementation took it at its rounding). */
void oracle_gat_bwd(int32_t n, const int32_t* indptr, const int32_t* indices,
                    int32_t f_in, int32_t h, const double* X, const double* W,
                    const double* a, double alpha, const double* Y,
                    const double* dY, double* dX, double* dW, double* da,
                    const uint8_t* z_pos) {
  const size_t nh = (size_t)n * (size_t)h;
  double* P = (double*)malloc(sizeof(double) * (nh ? nh : 1));
  double* G = (double*)malloc(sizeof(double) * (nh ? nh : 1));
  double* dP = (double*)calloc(nh ? nh : 1, sizeof(double));
  oracle_mm_nn(n, h, f_in, X, W, P);
  mask_all((int64_t)nh, Y, dY, G);
  for (int32_t c = 0; c < 2 * h; ++c) da[c] = 0.0;
  for (int32_t u = 0; u < n; ++u)
    for (int32_t j = indptr[u]; j < indptr[u + 1]; ++j) {
      const int32_t v = indices[j];
      const double* Pu = P + (int64_t)u * h;
      const double* Pv = P + (int64_t)v * h;
      const double* Gu = G + (int64_t)u * h;
      double z = 0.0, dA = 0.0;
      for (int32_t c = 0; c < h; ++c) z += a[c] * Pu[c] + a[h + c] * Pv[c];
      const int pos = z_pos ? (z_pos[j] != 0) : (z > 0.0);
      const double att = pos ? z : alpha * z;
      for (int32_t c = 0; c < h; ++c) dA += Gu[c] * Pv[c];
      const double dz = dA * (pos ? 1.0 : alpha);
      for (int32_t c = 0; c < h; ++c) {
        dP[(int64_t)v * h + c] += att * Gu[c];      /* A_att^T G */
        dP[(int64_t)u * h + c] += dz * a[c];        /* through a1 . P_u */
        dP[(int64_t)v * h + c] += dz * a[h + c];    /* through a2 . P_v */
        da[c] += dz * Pu[c];
        da[h + c] += dz * Pv[c];
      }
    }
  oracle_mm_tn(f_in, h, n, X, dP, dW);
  if (dX) oracle_mm_nt(n, f_in, h, dP, W, dX);
  free(dP);
  free(G);
  free(P);
}

/* ------------------------------------- classifier, loss and weight update */

/* Section 3.1 (Eqs. "mlp forward", "loss forward") and Algorithm 1:
 *   Z = X W  (n x C),  X_MLP = ReLU(Z),  Y = sigma(X_MLP)
 * sigma: kind 0 = row-wise softmax, kind 1 = element-wise sigmoid.
 *   L = (1/n) sum_v CE(Y_v, T_v): softmax  -sum_c T log Y,
 *                                  sigmoid -sum_c [T log Y + (1-T) log(1-Y)]
 * Section 5.1: dL/dX_MLP = (Y - T) / n;  G = that * 1[X_MLP > 0] (the MLP's
 * ReLU);  dW = X^T G;  dX = G W^T.  probs, dX may be NULL.  Returns L.
 * relu_on (n x C, may be NULL) supplies the ReLU's decision instead of
 * Z > 0: X_MLP = Z where it is 1, else 0, and the derivative is relu_on
 * (the decision another implementation took at its own rounding). */
double oracle_classifier(int32_t n, int32_t f, int32_t C, const double* X,
                         const double* W, const double* T, int32_t kind,
                         double* probs, double* dW, double* dX,
                         const uint8_t* relu_on) {
  const size_t nc = (size_t)n * (size_t)C;
  double* Z = (double*)malloc(sizeof(double) * (nc ? nc : 1));
  double* G = (double*)malloc(sizeof(double) * (nc ? nc : 1));
  oracle_mm_nn(n, C, f, X, W, Z);
  /* Z becomes X_MLP; `on` keeps the ReLU's derivative */
  uint8_t* on = (uint8_t*)malloc(nc ? nc : 1);
  for (size_t i = 0; i < nc; ++i) {
    on[i] = relu_on ? (relu_on[i] != 0) : (Z[i] > 0.0);
    Z[i] = on[i] ? Z[i] : 0.0;
  }
  double loss = 0.0;
  for (int64_t v = 0; v < n; ++v) {
    const double* z = Z + v * C;
    const double* t = T + v * C;
    double* g = G + v * C;
    double row = 0.0;
    if (kind == 0) {
      double m = z[0];
      for (int32_t c = 1; c < C; ++c) m = z[c] > m ? z[c] : m;
      double s = 0.0;
      for (int32_t c = 0; c < C; ++c) s += exp(z[c] - m);
      for (int32_t c = 0; c < C; ++c) {
        const double lp = z[c] - m - log(s); /* log Y */
        const double y = exp(lp);
        row -= t[c] * lp;
        g[c] = y;
      }
    } else {
      for (int32_t c = 0; c < C; ++c) {
        const double x = z[c];
        const double y = 1.0 / (1.0 + exp(-x));
        /* log Y = -log(1 + e^-x), log(1-Y) = -x - log(1 + e^-x) */
        const double l1 = -log1p(exp(-x));
        row -= t[c] * l1 + (1.0 - t[c]) * (l1 - x);
        g[c] = y;
      }
    }
    loss += row;
    for (int32_t c = 0; c < C; ++c) {
      if (probs) probs[v * C + c] = g[c];
      g[c] = on[v * C + c] ? (g[c] - t[c]) / (double)n : 0.0;
    }
  }
  oracle_mm_tn(f, C, n, X, G, dW);
  if (dX) oracle_mm_nt(n, f, C, G, W, dX);
  free(on);
  free(Z);
  free(G);
  return loss / (double)n;
}

/* Weight update by the gradient (Algorithm 1): W -= lr g. */
void oracle_sgd(int64_t count, double* W, const double* g, double lr) {
  for (int64_t i = 0; i < count; ++i) W[i] -= lr * g[i];
}

/* Adam (Algorithm 1 leaves the update rule open; Adam is offered beside
 * plain gradient descent): step t >= 1,
 *   m = b1 m + (1-b1) g;  v = b2 v + (1-b2) g^2;
 *   W -= lr (m / (1 - b1^t)) / (sqrt(v / (1 - b2^t)) + eps). */
void oracle_adam(int64_t count, double* W, const double* g, double* m,
                 double* v, double lr, double b1, double b2, double eps,
                 int32_t t) {
  const double c1 = 1.0 - pow(b1, t), c2 = 1.0 - pow(b2, t);
  for (int64_t i = 0; i < count; ++i) {
    m[i] = b1 * m[i] + (1.0 - b1) * g[i];
    v[i] = b2 * v[i] + (1.0 - b2) * g[i] * g[i];
    W[i] -= lr * (m[i] / c1) / (sqrt(v[i] / c2) + eps);
  }
}

/* ------------------------------------------------ induced subgraph (prep) */

static int cmp_i32(const void* a, const void* b) {
  const int32_t x = *(const int32_t*)a, y = *(const int32_t*)b;
  return (x > y) - (x < y);
}

/* Position of w in the sorted list nodes[0..n_s), or -1. */
static int32_t find_node(int32_t n_s, const int32_t* nodes, int32_t w) {
  int32_t lo = 0, hi = n_s;
  while (lo < hi) {
    const int32_t mid = lo + (hi - lo) / 2;
    if (nodes[mid] < w) lo = mid + 1; else hi = mid;
  }
  return (lo < n_s && nodes[lo] == w) ? lo : -1;
}

/* Algorithm 2's last step and Algorithm 1's "adjacency matrix of G_s": the
 * subgraph of the full graph induced by V_s = nodes (sorted, distinct;
 * nodes[i] becomes node i), every node with its self loop, then the
 * normalisation of Eq. "graphsage forward", D^-1 A with D counting the
 * stored entries (norm 0: each entry of row u is 1/len_u), or the
 * symmetric one of the GCN layer (norm 1: 1/sqrt(len_u len_v)).  Rows come
 * out sorted.  out_indices / out_values need room for the sum over V_s of
 * (full degree + 1).  Returns the number of stored entries. */
int64_t oracle_induce(int64_t n_full, const int64_t* indptr,
                      const int32_t* indices, int32_t n_s,
                      const int32_t* nodes, int32_t norm, int32_t* out_indptr,
                      int32_t* out_indices, double* out_values) {
  (void)n_full;
  int64_t nnz = 0;
  out_indptr[0] = 0;
  for (int32_t i = 0; i < n_s; ++i) {
    const int32_t v = nodes[i];
    int32_t* row = out_indices + nnz;
    int32_t len = 0;
    row[len++] = i; /* the self loop */
    for (int64_t j = indptr[v]; j < indptr[v + 1]; ++j) {
      const int32_t w = indices[j];
      if (w == v) continue; /* a stored loop of the full graph counts once */
      const int32_t k = find_node(n_s, nodes, w);
      if (k >= 0) row[len++] = k;
    }
    qsort(row, (size_t)len, sizeof(int32_t), cmp_i32);
    nnz += len;
    out_indptr[i + 1] = (int32_t)nnz;
  }
  for (int32_t i = 0; i < n_s; ++i) {
    const int32_t lu = out_indptr[i + 1] - out_indptr[i];
    for (int32_t j = out_indptr[i]; j < out_indptr[i + 1]; ++j) {
      const int32_t k = out_indices[j];
      const int32_t lv = out_indptr[k + 1] - out_indptr[k];
      out_values[j] = norm == 0 ? 1.0 / (double)lu : 1.0 / sqrt((double)lu * (double)lv);
    }
  }
  return nnz;
}

/* ---------------------------------------------- per-output spot evaluation */

void oracle_sage_fwd_rows(int32_t n, const int32_t* indptr,
                          const int32_t* indices, const double* values,
                          int32_t f_in, int32_t h, const double* X,
                          const double* W_self, const double* W_neigh,
                          const double* b_self, const double* b_neigh,
                          int32_t nrows, const int32_t* rows, double* Y_rows) {
  (void)n;
#pragma omp parallel for schedule(dynamic, 1)
  for (int32_t r = 0; r < nrows; ++r) {
    const int32_t v = rows[r];
    double* s = (double*)malloc(sizeof(double) * (size_t)(f_in > 0 ? f_in : 1));
    for (int32_t k = 0; k < f_in; ++k) s[k] = 0.0;
    for (int32_t j = indptr[v]; j < indptr[v + 1]; ++j)
      for (int32_t k = 0; k < f_in; ++k)
        s[k] += values[j] * X[(int64_t)indices[j] * f_in + k];
    for (int32_t c = 0; c < h; ++c) {
      double zs = 0.0, zn = 0.0;
      for (int32_t k = 0; k < f_in; ++k) {
        zs += X[(int64_t)v * f_in + k] * W_self[(int64_t)k * h + c];
        zn += s[k] * W_neigh[(int64_t)k * h + c];
      }
      if (b_self) zs += b_self[c];
      if (b_neigh) zn += b_neigh[c];
      Y_rows[(int64_t)r * 2 * h + c] = relu(zs);
      Y_rows[(int64_t)r * 2 * h + h + c] = relu(zn);
    }
    free(s);
  }
}

void oracle_sage_bwd_dx_rows(int32_t n, const int32_t* indptr,
                             const int32_t* indices, const double* values,
                             int32_t f_in, int32_t h, const double* W_self,
                             const double* W_neigh, const double* Y,
                             const double* dY, int32_t nrows,
                             const int32_t* rows, double* dX_rows) {
#pragma omp parallel for schedule(dynamic, 1)
  for (int32_t r = 0; r < nrows; ++r) {
    const int32_t u = rows[r];
    /* t = row u of (A_s)^T G_n: every stored (v,u), v ascending. */
    double* t = (double*)malloc(sizeof(double) * (size_t)(h > 0 ? h : 1));
    for (int32_t c = 0; c < h; ++c) t[c] = 0.0;
    for (int32_t v = 0; v < n; ++v)
      for (int32_t j = indptr[v]; j < indptr[v + 1]; ++j)
        if (indices[j] == u)
          for (int32_t c = 0; c < h; ++c) {
            const int64_t b = (int64_t)v * 2 * h + h + c;
            t[c] += values[j] * (Y[b] > 0.0 ? dY[b] : 0.0);
          }
    for (int32_t k = 0; k < f_in; ++k) {
      double a = 0.0, b = 0.0;
      for (int32_t c = 0; c < h; ++c) {
        const int64_t s = (int64_t)u * 2 * h + c;
        a += (Y[s] > 0.0 ? dY[s] : 0.0) * W_self[(int64_t)k * h + c];
        b += t[c] * W_neigh[(int64_t)k * h + c];
      }
      dX_rows[(int64_t)r * f_in + k] = a + b;
    }
    free(t);
  }
}

void oracle_sage_bwd_dw_entries(int32_t n, const int32_t* indptr,
                                const int32_t* indices, const double* values,
                                int32_t f_in, int32_t h, const double* X,
                                const double* Y, const double* dY,
                                int32_t nent, const int32_t* ei,
                                const int32_t* ej, double* dWs_ent,
                                double* dWn_ent) {
#pragma omp parallel for schedule(dynamic, 1)
  for (int32_t e = 0; e < nent; ++e) {
    const int32_t i = ei[e], c = ej[e];
    double ws = 0.0, wn = 0.0;
    for (int32_t v = 0; v < n; ++v) {
      const int64_t a = (int64_t)v * 2 * h + c, b = a + h;
      double s = 0.0; /* (A_s X)[v, i] */
      for (int32_t j = indptr[v]; j < indptr[v + 1]; ++j)
        s += values[j] * X[(int64_t)indices[j] * f_in + i];
      ws += X[(int64_t)v * f_in + i] * (Y[a] > 0.0 ? dY[a] : 0.0);
      wn += s * (Y[b] > 0.0 ? dY[b] : 0.0);
    }
    dWs_ent[e] = ws;
    dWn_ent[e] = wn;
  }
}
