// C-ABI of libgnnprop: argument checks, workspace carving and the launch
// sequence of one GraphSAGE layer's forward and backward pass.
//
// Forward (Section 2.1, Eq. "graphsage forward"), with the Section 6.1
// order choice for the neighbour path A_s X W_neigh:
//   order 1:  S = A_s X (kept for the backward pass)
//             [Y_self | Y_neigh] = ReLU([X W_self + b_s | S W_neigh + b_n])
//             -- one aggregation, one two-problem matrix-core launch
//   order 2:  [Y_self | P] = [ReLU(X W_self + b_s) | X W_neigh]
//             Y_neigh = ReLU(A_s P + b_n)   (bias + ReLU fused into the
//                                            aggregation's store)
// Backward (Section 5.1, Eq. "gcn backward"), G = dY * 1[Y > 0]:
//   order 2:  [G_s | G_n] <- mask;  T = (A_s)^T G_n
//             dW_self = X^T G_s, dW_neigh = X^T T     ( = (A_s X)^T G_n )
//             dX = G_s W_self^T + T W_neigh^T         (one launch, 2 K parts)
//   order 1:  G <- mask;  dW_self = X^T G_s, dW_neigh = S^T G_n
//             dX = G_s W_self^T;  V = G_n W_neigh^T;  dX += (A_s)^T V
#include <algorithm>
#include <cstring>
#include <vector>

#include "abi.hpp"

using namespace gnnprop;

namespace {

// ------------------------------------------------------------- timer

struct TimerRec {
  int kclass;
  double work;
  hipEvent_t a, b;
};
bool g_timer_on = false;
std::vector<hipEvent_t> g_pool;
size_t g_pool_used = 0;
std::vector<TimerRec> g_recs;
TimerRec g_cur;

// ------------------------------------------------------- layer layout

struct LayerLayout {
  int order;
  int64_t ld_s, ld_p, ld_g, ld_gn, ld_v;
  // bf16 products, order 2: G_s and T as bf16 (row stride ld_h16) in buf0,
  // T at off_t16 bytes past G_s
  int64_t ld_h16;
  size_t off_t16;
  size_t wp_words;  // split products: words of one weight's bf16 pieces
  // GEMM workspace: [off_gemm, off_gemm_x) holds the weight gradients'
  // partial tiles, which stay there until the input-gradient launch that
  // follows sums them; [off_gemm_x, off_cs) serves every other launch
  size_t off_buf0, off_buf1, off_gemm, off_gemm_x, off_cs, off_wp, total;
  // saved buffer: order 1's A_s X (n x ld_s floats) at 0; with split
  // products the input gradient's pieces of W_self^T and W_neigh^T (sp_words
  // words each, K = h, N = f_in), written by the forward's weight split, at
  // off_sp and off_sp + sp_stride
  size_t sp_words, off_sp, sp_stride, saved_total;
};

int resolve_order(const gnn_layer* L) {
  return L->order ? L->order : gnn_choose_order(L->f_in, L->h);
}

GemmBatch fwd_batch(int order, int32_t n, int32_t f_in, int32_t h,
                    const float* X, int64_t ld_x, const float* S, int64_t ld_s,
                    const float* Ws, const float* Wn, const float* bs,
                    const float* bn, float* Y, int64_t ld_y, float* P,
                    int64_t ld_p) {
  GemmBatch b;
  memset(&b, 0, sizeof(b));
  b.nprob = 2;
  b.trans_a = 0;
  b.trans_b = 0;
  GemmProblem& p0 = b.p[0];
  p0.nseg = 1;
  p0.seg[0] = {X, Ws, ld_x, h, f_in};
  p0.M = n;
  p0.N = h;
  p0.C = Y;
  p0.ldc = ld_y;
  p0.bias = bs;
  p0.relu = 1;
  GemmProblem& p1 = b.p[1];
  p1.nseg = 1;
  p1.M = n;
  p1.N = h;
  if (order == 1) {  // Y_neigh = ReLU(S W_neigh + b_n)
    p1.seg[0] = {S, Wn, ld_s, h, f_in};
    p1.C = Y ? Y + h : nullptr;
    p1.ldc = ld_y;
    p1.bias = bn;
    p1.relu = 1;
  } else {           // P = X W_neigh
    p1.seg[0] = {X, Wn, ld_x, h, f_in};
    p1.C = P;
    p1.ldc = ld_p;
    p1.bias = nullptr;
    p1.relu = 0;
  }
  return b;
}

// dW_self = X^T G_s ; dW_neigh = (order 1: S, order 2: X)^T (G_n or T)
GemmBatch dw_batch(int order, int32_t n, int32_t f_in, int32_t h,
                   const float* X, int64_t ld_x, const float* S, int64_t ld_s,
                   const float* Gs, int64_t ld_gs, const float* Gn,
                   int64_t ld_gn, float* dWs, float* dWn) {
  GemmBatch b;
  memset(&b, 0, sizeof(b));
  b.nprob = 2;
  b.trans_a = 1;
  b.trans_b = 0;
  for (int i = 0; i < 2; ++i) {
    GemmProblem& p = b.p[i];
    p.nseg = 1;
    p.M = f_in;
    p.N = h;
    p.ldc = h;
    p.relu = 0;
    p.bias = nullptr;
  }
  b.p[0].seg[0] = {X, Gs, ld_x, ld_gs, n};
  b.p[0].C = dWs;
  if (order == 1)
    b.p[1].seg[0] = {S, Gn, ld_s, ld_gn, n};
  else
    b.p[1].seg[0] = {X, Gn, ld_x, ld_gn, n};
  b.p[1].C = dWn;
  return b;
}

// order 2: dX = G_s W_s^T + T W_n^T (one problem, two K parts)
// order 1: dX = G_s W_s^T ; V = G_n W_n^T
GemmBatch dx_batch(int order, int32_t n, int32_t f_in, int32_t h,
                   const float* Gs, int64_t ld_gs, const float* Gn,
                   int64_t ld_gn, const float* Ws, const float* Wn, float* dX,
                   int64_t ld_dx, float* V, int64_t ld_v) {
  GemmBatch b;
  memset(&b, 0, sizeof(b));
  b.trans_a = 0;
  b.trans_b = 1;
  if (order == 2) {
    b.nprob = 1;
    GemmProblem& p = b.p[0];
    p.nseg = 2;
    p.seg[0] = {Gs, Ws, ld_gs, h, h};
    p.seg[1] = {Gn, Wn, ld_gn, h, h};
    p.M = n;
    p.N = f_in;
    p.C = dX;
    p.ldc = ld_dx;
  } else {
    b.nprob = 2;
    for (int i = 0; i < 2; ++i) {
      b.p[i].nseg = 1;
      b.p[i].M = n;
      b.p[i].N = f_in;
    }
    b.p[0].seg[0] = {Gs, Ws, ld_gs, h, h};
    b.p[0].C = dX;
    b.p[0].ldc = ld_dx;
    b.p[1].seg[0] = {Gn, Wn, ld_gn, h, h};
    b.p[1].C = V;
    b.p[1].ldc = ld_v;
  }
  return b;
}

// Split products: W_self and W_neigh pre-split into their bf16 pieces in
// the workspace (once per call, in the orientation of this batch's B), and
// the batch's segments pointed at them: segment B pointers equal to W_self
// take the first, W_neigh the second.
// Points the batch's weight segments at bf16 pieces: p_self for W_self's,
// p_neigh for W_neigh's, pw words per plane.
void use_weight_planes(GemmBatch& b, const float* Ws, const uint32_t* p_self,
                       const uint32_t* p_neigh, int64_t pw) {
  for (int i = 0; i < b.nprob; ++i)
    for (int k = 0; k < b.p[i].nseg; ++k) {
      GemmSeg& sg = b.p[i].seg[k];
      sg.Bp = sg.B == Ws ? p_self : p_neigh;
      sg.bp_plane = pw;
    }
  b.b_planes = 1;
}

// The input gradient's pieces in the saved buffer: i = 0 W_self's, 1 W_neigh's.
uint32_t* saved_plane(const LayerLayout& o, void* saved, int i) {
  return reinterpret_cast<uint32_t*>(static_cast<char*>(saved) + o.off_sp + i * o.sp_stride);
}
const uint32_t* saved_plane(const LayerLayout& o, const void* saved, int i) {
  return reinterpret_cast<const uint32_t*>(static_cast<const char*>(saved) + o.off_sp +
                                           i * o.sp_stride);
}

// Forward product (split products): W_self and W_neigh split once into the
// workspace in the forward orientation (op(B) = W, K = f_in, N = h) and, in
// the same launch, into the saved buffer in the input gradient's (op(B) =
// W^T, K = h, N = f_in), which gnn_prop_bwd reads instead of splitting.
hipError_t attach_weight_planes(GemmBatch& b, const LayerLayout& o, char* ws, void* saved,
                                const float* Ws, const float* Wn, int32_t f_in,
                                int32_t h, hipStream_t s) {
  if (b.mode != GEMM_SPLIT) return hipSuccess;
  uint32_t* wp[2] = {reinterpret_cast<uint32_t*>(ws + o.off_wp),
                     reinterpret_cast<uint32_t*>(ws + o.off_wp + round_up(o.wp_words * 4, 256))};
  const SplitJob jobs[4] = {{Ws, h, f_in, h, 0, wp[0]},
                            {Wn, h, f_in, h, 0, wp[1]},
                            {Ws, h, h, f_in, 1, saved_plane(o, saved, 0)},
                            {Wn, h, h, f_in, 1, saved_plane(o, saved, 1)}};
  hipError_t e = split_b_planes_launch(jobs, 4, s);
  if (e != hipSuccess) return e;
  use_weight_planes(b, Ws, wp[0], wp[1], (int64_t)(b_planes_words(f_in, h) / 3));
  return hipSuccess;
}

GemmBatch with_mode(GemmBatch b, int32_t mode) {
  b.mode = mode;
  return b;
}

LayerLayout layer_layout(const gnn_csr* csr, const gnn_layer* L) {
  LayerLayout o;
  const int32_t n = csr->n, f_in = L->f_in, h = L->h;
  o.order = resolve_order(L);
  o.ld_s = round_up(f_in, 4);
  o.ld_p = round_up(h, 4);
  o.ld_g = round_up(2 * (int64_t)h, 4);
  o.ld_gn = round_up(h, 4);
  o.ld_v = round_up(f_in, 4);
  size_t buf0, buf1;
  o.ld_h16 = round_up(h, 4);
  o.off_t16 = round_up((size_t)n * o.ld_h16 * 2, 256);
  if (o.order == 2) {
    buf0 = std::max((size_t)n * o.ld_p, (size_t)n * o.ld_g) * 4;  // P | GT
    if (gemm_mode(L->flags) == GEMM_BF16) buf0 = std::max(buf0, 2 * o.off_t16);  // G_s, T bf16
    buf1 = (size_t)n * o.ld_gn * 4;                               // G_n
  } else {
    buf0 = (size_t)n * o.ld_g * 4;  // G
    buf1 = (size_t)n * o.ld_v * 4;  // V
  }
  const int32_t bf = gemm_mode(L->flags);
  const size_t gemm_w = gemm_workspace_bytes(with_mode(dw_batch(o.order, n, f_in, h, 0, f_in, 0, 0, 0, 2 * h, 0, 2 * h, 0, 0), bf));
  const size_t gemm = std::max(
      gemm_workspace_bytes(with_mode(fwd_batch(o.order, n, f_in, h, 0, f_in, 0, 0, 0, 0, 0, 0, 0, 2 * h, 0, 0), bf)),
      gemm_workspace_bytes(with_mode(dx_batch(o.order, n, f_in, h, 0, 2 * h, 0, 2 * h, 0, 0, 0, f_in, 0, f_in), bf)));
  // split products: W_self and W_neigh as bf16 pieces in the forward
  // product's orientation (K = f_in, N = h) in the workspace; the input
  // gradient's (K = h, N = f_in) in the saved buffer
  o.wp_words = bf == GEMM_SPLIT ? b_planes_words(f_in, h) : 0;
  o.sp_words = bf == GEMM_SPLIT ? b_planes_words(h, f_in) : 0;
  o.off_sp = o.order == 1 ? round_up((size_t)n * o.ld_s * 4, 256) : 0;
  o.sp_stride = round_up(o.sp_words * 4, 256);
  o.saved_total = o.off_sp + 2 * o.sp_stride;
  o.off_buf0 = 0;
  o.off_buf1 = round_up(buf0, 256);
  o.off_gemm = o.off_buf1 + round_up(buf1, 256);
  o.off_gemm_x = o.off_gemm + round_up(gemm_w, 256);
  o.off_cs = o.off_gemm_x + round_up(gemm, 256);
  o.off_wp = o.off_cs + round_up(colsum_partials_bytes(n, h), 256);
  o.total = o.off_wp + 2 * round_up(o.wp_words * 4, 256);
  return o;
}

gnn_status check_layer(const gnn_layer* L) {
  if (!L) return GNN_ERR_NULL;
  if (L->f_in <= 0 || L->h <= 0) return GNN_ERR_SHAPE;
  if (L->ld_x < L->f_in || L->ld_y < 2 * (int64_t)L->h) return GNN_ERR_SHAPE;
  if (L->order < 0 || L->order > 2) return GNN_ERR_SHAPE;
  if ((L->flags & ~(GEMM_FLAGS | GNN_FLAG_DY_MASKED | GNN_FLAG_DX_MASKED |
                    GNN_FLAG_ROW_NORMALIZED)) ||
      !gemm_flags_ok(L->flags))
    return GNN_ERR_UNSUPPORTED;
  return GNN_OK;
}

}  // namespace

namespace gnnprop {

void timer_begin(int kclass, hipStream_t s) {
  if (!g_timer_on) return;
  while (g_pool_used + 2 > g_pool.size()) {
    hipEvent_t e;
    if (hipEventCreate(&e) != hipSuccess) return;
    g_pool.push_back(e);
  }
  g_cur.kclass = kclass;
  g_cur.a = g_pool[g_pool_used++];
  g_cur.b = g_pool[g_pool_used++];
  (void)hipEventRecord(g_cur.a, s);
}

void timer_end(int kclass, double work, hipStream_t s) {
  if (!g_timer_on || g_cur.kclass != kclass) return;
  (void)hipEventRecord(g_cur.b, s);
  g_cur.work = work;
  g_recs.push_back(g_cur);
  g_cur.kclass = -1;
}

}  // namespace gnnprop

extern "C" {

const char* gnn_status_string(gnn_status s) {
  switch (s) {
    case GNN_OK: return "ok";
    case GNN_ERR_NULL: return "required pointer is NULL";
    case GNN_ERR_SHAPE: return "invalid size or leading dimension";
    case GNN_ERR_CSR: return "invalid CSR";
    case GNN_ERR_UNSUPPORTED: return "unsupported option";
    case GNN_ERR_WORKSPACE: return "workspace or plan buffer too small";
    case GNN_ERR_HIP: return "HIP runtime error";
    case GNN_ERR_ALIAS: return "output overlaps an input";
  }
  return "unknown status";
}

int32_t gnn_choose_order(int32_t f_in, int32_t h) { return f_in <= h ? 1 : 2; }

size_t gnn_plan_bytes(int32_t n, int64_t nnz) {
  if (n < 0 || nnz < 0) return 0;
  return plan_dims(n, nnz).bytes;
}

gnn_status gnn_csr_transpose_values(const gnn_csr* csr, float* values_t,
                                    hipStream_t stream) {
  gnn_status st = check_csr(csr, true, false);
  if (st != GNN_OK) return st;
  if (csr->nnz > 0 && !values_t) return GNN_ERR_NULL;
  if (ranges_overlap(values_t, csr->nnz * 4, csr->values, csr->nnz * 4))
    return GNN_ERR_ALIAS;
  GNN_HIP(transpose_values_launch(csr->n, csr->nnz, csr->indptr, csr->indices,
                                  csr->values, values_t, csr->plan, stream));
  return GNN_OK;
}

gnn_status gnn_csr_build_plan(const gnn_csr* csr, void* plan,
                              size_t plan_bytes, hipStream_t stream) {
  gnn_status st = check_csr(csr, false, false);
  if (st != GNN_OK) return st;
  if (!plan) return GNN_ERR_NULL;
  if (!buf16(plan)) return GNN_ERR_UNSUPPORTED;
  if (plan_bytes < gnn_plan_bytes(csr->n, csr->nnz)) return GNN_ERR_WORKSPACE;
  GNN_HIP(plan_build_launch(csr->n, csr->nnz, csr->indptr, csr->indices,
                            plan, stream));
  return GNN_OK;
}

gnn_status gnn_csr_prepare(const gnn_csr* csr, void* plan, size_t plan_bytes,
                           float* values_t, hipStream_t stream) {
  gnn_status st = check_csr(csr, true, false);
  if (st != GNN_OK) return st;
  if (!plan) return GNN_ERR_NULL;
  if (csr->nnz > 0 && !values_t) return GNN_ERR_NULL;
  if (!buf16(plan)) return GNN_ERR_UNSUPPORTED;
  if (plan_bytes < gnn_plan_bytes(csr->n, csr->nnz)) return GNN_ERR_WORKSPACE;
  const size_t vb = (size_t)csr->nnz * 4;
  if (ranges_overlap(values_t, vb, csr->values, vb) ||
      ranges_overlap(plan, plan_bytes, values_t, vb) ||
      ranges_overlap(plan, plan_bytes, csr->values, vb) ||
      ranges_overlap(plan, plan_bytes, csr->indptr, ((size_t)csr->n + 1) * 4) ||
      ranges_overlap(plan, plan_bytes, csr->indices, (size_t)csr->nnz * 4))
    return GNN_ERR_ALIAS;
  GNN_HIP(prepare_launch(csr->n, csr->nnz, csr->indptr, csr->indices, csr->values,
                         values_t, plan, stream));
  return GNN_OK;
}

gnn_status gnn_csr_validate(const gnn_csr* csr, int32_t require_symmetric,
                            hipStream_t stream) {
  gnn_status st = check_csr(csr, false, false);
  if (st != GNN_OK) return st;
  int32_t* bad = nullptr;
  GNN_HIP(hipMalloc(&bad, sizeof(int32_t)));
  int32_t h_bad = 0;
  hipError_t e = hipMemcpyAsync(bad, &h_bad, sizeof(int32_t),
                                hipMemcpyHostToDevice, stream);
  if (e == hipSuccess)
    e = validate_csr(csr->n, csr->nnz, csr->indptr, csr->indices,
                     require_symmetric, bad, stream);
  if (e == hipSuccess)
    e = hipMemcpyAsync(&h_bad, bad, sizeof(int32_t), hipMemcpyDeviceToHost,
                       stream);
  if (e == hipSuccess) e = hipStreamSynchronize(stream);
  (void)hipFree(bad);
  if (e != hipSuccess) return GNN_ERR_HIP;
  return h_bad ? GNN_ERR_CSR : GNN_OK;
}

size_t gnn_spmm_workspace_bytes(const gnn_csr* csr, int32_t w) {
  if (!csr || csr->n < 0 || csr->nnz < 0 || w < 0) return 0;
  return spmm_partials_bytes(csr->n, csr->nnz, w);
}

gnn_status gnn_spmm(const gnn_csr* csr, int32_t transpose, int32_t w,
                    const float* in, int64_t ld_in, float* out,
                    int64_t ld_out, void* workspace, size_t workspace_bytes,
                    hipStream_t stream) {
  gnn_status st = check_csr(csr, !transpose, transpose != 0);
  if (st != GNN_OK) return st;
  if (w < 0 || ld_in < w || ld_out < w) return GNN_ERR_SHAPE;
  if (csr->n == 0 || w == 0) return GNN_OK;
  if (!in || !out || !csr->plan) return GNN_ERR_NULL;
  if (!buf16(workspace)) return GNN_ERR_UNSUPPORTED;
  const size_t need = spmm_partials_bytes(csr->n, csr->nnz, w);
  if (workspace_bytes < need || (need > 0 && !workspace))
    return GNN_ERR_WORKSPACE;
  if (ranges_overlap(in, mat_bytes(csr->n, w, ld_in), out,
                     mat_bytes(csr->n, w, ld_out)))
    return GNN_ERR_ALIAS;
  SpmmCall c = spmm_call(csr, transpose != 0, w, in, ld_in, out, ld_out);
  GNN_HIP(spmm_launch(c, stream));
  return GNN_OK;
}

gnn_status gnn_spmm_gather_floor(const gnn_csr* csr, int32_t transpose,
                                 int32_t w, const float* in, int64_t ld_in,
                                 float* out, int64_t ld_out, hipStream_t stream) {
  gnn_status st = check_csr(csr, !transpose, transpose != 0);
  if (st != GNN_OK) return st;
  if (w < 0 || ld_in < w || ld_out < w) return GNN_ERR_SHAPE;
  if (csr->n == 0 || w == 0) return GNN_OK;
  if (!in || !out || !csr->plan) return GNN_ERR_NULL;
  if (!vec4_ok(in, ld_in) || !vec4_ok(out, ld_out)) return GNN_ERR_UNSUPPORTED;
  if (ranges_overlap(in, mat_bytes(csr->n, w, ld_in), out,
                     mat_bytes(csr->n, w, ld_out)))
    return GNN_ERR_ALIAS;
  SpmmCall c = spmm_call(csr, transpose != 0, w, in, ld_in, out, ld_out);
  GNN_HIP(spmm_floor_launch(c, stream));
  return GNN_OK;
}

// Split products pre-split B into its bf16 pieces once (workspace, after
// the partial tiles) when at least four row tiles of 128 share it: each
// would otherwise split the same values again.
static bool gemm_presplit_b(int32_t M, int32_t mode) {
  return mode == GEMM_SPLIT && M >= 512;
}

size_t gnn_gemm_workspace_bytes(int32_t M, int32_t N, int32_t K) {
  if (M < 0 || N < 0 || K < 0) return 0;
  GemmBatch b;
  memset(&b, 0, sizeof(b));
  b.nprob = 1;
  b.p[0].nseg = 1;
  b.p[0].M = M;
  b.p[0].N = N;
  b.p[0].seg[0].K = K;
  // the largest need of the three product modes (their work splits differ)
  size_t need = 0;
  for (const int32_t mode : {GEMM_SPLIT, GEMM_BF16, GEMM_F32}) {
    b.mode = mode;
    need = std::max(need, gemm_workspace_bytes(b));
  }
  const size_t part = round_up(need, 256);
  return part + (gemm_presplit_b(M, GEMM_SPLIT) ? round_up(b_planes_words(K, N) * 4, 256) : 0);
}

gnn_status gnn_gemm(int32_t trans_a, int32_t trans_b, int32_t M, int32_t N,
                    int32_t K, const float* A, int64_t lda, const float* B,
                    int64_t ldb, float* C, int64_t ldc, uint32_t flags,
                    void* workspace, size_t workspace_bytes,
                    hipStream_t stream) {
  if (M < 0 || N < 0 || K < 0) return GNN_ERR_SHAPE;
  if ((flags & ~GEMM_FLAGS) || !gemm_flags_ok(flags)) return GNN_ERR_UNSUPPORTED;
  if (M == 0 || N == 0) return GNN_OK;
  if (!C || (K > 0 && (!A || !B))) return GNN_ERR_NULL;
  if (ldc < N) return GNN_ERR_SHAPE;
  if (K > 0) {
    if (trans_a ? lda < M : lda < K) return GNN_ERR_SHAPE;
    if (trans_b ? ldb < K : ldb < N) return GNN_ERR_SHAPE;
  }
  if (!buf16(workspace)) return GNN_ERR_UNSUPPORTED;
  GemmBatch b;
  memset(&b, 0, sizeof(b));
  b.nprob = 1;
  b.trans_a = trans_a != 0;
  b.trans_b = trans_b != 0;
  b.mode = gemm_mode(flags);
  b.p[0].nseg = 1;
  b.p[0].seg[0] = {A, B, lda, ldb, K};
  b.p[0].M = M;
  b.p[0].N = N;
  b.p[0].C = C;
  b.p[0].ldc = ldc;
  const size_t part = round_up(gemm_workspace_bytes(b), 256);
  const bool presplit = K > 0 && gemm_presplit_b(M, b.mode);
  const size_t need = part + (presplit ? round_up(b_planes_words(K, N) * 4, 256) : 0);
  if (workspace_bytes < need || (need > 0 && !workspace))
    return GNN_ERR_WORKSPACE;
  const size_t cb = mat_bytes(M, N, ldc);
  if (K > 0 &&
      (ranges_overlap(C, cb, A, trans_a ? mat_bytes(K, M, lda) : mat_bytes(M, K, lda)) ||
       ranges_overlap(C, cb, B, trans_b ? mat_bytes(N, K, ldb) : mat_bytes(K, N, ldb))))
    return GNN_ERR_ALIAS;
  if (presplit) {
    uint32_t* planes = reinterpret_cast<uint32_t*>(static_cast<char*>(workspace) + part);
    const SplitJob job = {B, ldb, K, N, trans_b != 0, planes};
    GNN_HIP(split_b_planes_launch(&job, 1, stream));
    b.b_planes = 1;
    b.p[0].seg[0].Bp = planes;
    b.p[0].seg[0].bp_plane = (int64_t)(b_planes_words(K, N) / 3);
  }
  GNN_HIP(gemm_launch(b, workspace, part, stream));
  return GNN_OK;
}

size_t gnn_prop_saved_bytes(const gnn_csr* csr, const gnn_layer* layer) {
  if (!csr || !layer || csr->n < 0 || csr->nnz < 0 || layer->f_in <= 0 || layer->h <= 0)
    return 0;
  return layer_layout(csr, layer).saved_total;
}

size_t gnn_prop_workspace_bytes(const gnn_csr* csr, const gnn_layer* layer) {
  if (!csr || !layer || csr->n < 0 || csr->nnz < 0 || layer->f_in <= 0 ||
      layer->h <= 0)
    return 0;
  return layer_layout(csr, layer).total;
}

gnn_status gnn_prop_fwd(const gnn_csr* csr, const gnn_layer* layer,
                        const float* X, const float* W_self,
                        const float* W_neigh, const float* b_self,
                        const float* b_neigh, float* Y, void* saved,
                        void* workspace, size_t workspace_bytes,
                        hipStream_t stream) {
  gnn_status st = check_layer(layer);
  if (st != GNN_OK) return st;
  const bool rn = (layer->flags & GNN_FLAG_ROW_NORMALIZED) != 0;
  if ((st = check_csr(csr, !rn, false)) != GNN_OK) return st;
  const int32_t n = csr->n, f_in = layer->f_in, h = layer->h;
  if (n > 0 && (!X || !Y || !csr->plan)) return GNN_ERR_NULL;
  if (!W_self || !W_neigh) return GNN_ERR_NULL;
  const LayerLayout o = layer_layout(csr, layer);
  if (o.saved_total > 0 && n > 0 && !saved) return GNN_ERR_NULL;
  if (!buf16(workspace) || !buf16(saved)) return GNN_ERR_UNSUPPORTED;
  if (workspace_bytes < o.total || (o.total > 0 && !workspace))
    return GNN_ERR_WORKSPACE;
  if (n == 0) return GNN_OK;
  const size_t yb = mat_bytes(n, 2 * h, layer->ld_y);
  if (ranges_overlap(Y, yb, X, mat_bytes(n, f_in, layer->ld_x)) ||
      ranges_overlap(Y, yb, W_self, (size_t)f_in * h * 4) ||
      ranges_overlap(Y, yb, W_neigh, (size_t)f_in * h * 4))
    return GNN_ERR_ALIAS;

  char* ws = static_cast<char*>(workspace);
  void* gws = ws + o.off_gemm;
  const size_t gws_bytes = o.off_cs - o.off_gemm;
  if (o.order == 1) {
    float* S = static_cast<float*>(saved);
    SpmmCall c = spmm_call(csr, false, f_in, X, layer->ld_x, S, o.ld_s, rn);
    GNN_HIP(spmm_launch(c, stream));
    GemmBatch b = fwd_batch(1, n, f_in, h, X, layer->ld_x, S, o.ld_s, W_self,
                            W_neigh, b_self, b_neigh, Y, layer->ld_y, nullptr, 0);
    b.mode = gemm_mode(layer->flags);
    GNN_HIP(attach_weight_planes(b, o, ws, saved, W_self, W_neigh, f_in, h, stream));
    GNN_HIP(gemm_launch(b, gws, gws_bytes, stream));
  } else {
    float* P = reinterpret_cast<float*>(ws + o.off_buf0);
    GemmBatch b = fwd_batch(2, n, f_in, h, X, layer->ld_x, nullptr, 0, W_self,
                            W_neigh, b_self, nullptr, Y, layer->ld_y, P, o.ld_p);
    b.mode = gemm_mode(layer->flags);
    GNN_HIP(attach_weight_planes(b, o, ws, saved, W_self, W_neigh, f_in, h, stream));
    GNN_HIP(gemm_launch(b, gws, gws_bytes, stream));
    SpmmCall c = spmm_call(csr, false, h, P, o.ld_p, Y + h, layer->ld_y, rn);
    c.epilogue = SPMM_BIAS_RELU;
    c.bias = b_neigh;
    GNN_HIP(spmm_launch(c, stream));
  }
  return GNN_OK;
}

gnn_status gnn_prop_bwd(const gnn_csr* csr, const gnn_layer* layer,
                        const float* X, const float* W_self,
                        const float* W_neigh, const float* Y, const float* dY,
                        const void* saved, float* dX, float* dW_self,
                        float* dW_neigh, float* db_self, float* db_neigh,
                        void* workspace, size_t workspace_bytes,
                        hipStream_t stream) {
  gnn_status st = check_layer(layer);
  if (st != GNN_OK) return st;
  const bool rn = (layer->flags & GNN_FLAG_ROW_NORMALIZED) != 0;
  if ((st = check_csr(csr, !rn, !rn)) != GNN_OK) return st;
  const int32_t n = csr->n, f_in = layer->f_in, h = layer->h;
  if (!W_self || !W_neigh || !dW_self || !dW_neigh) return GNN_ERR_NULL;
  if (n > 0 && (!X || !Y || !dY || !csr->plan)) return GNN_ERR_NULL;
  if (dX && layer->ld_dx < f_in) return GNN_ERR_SHAPE;
  const LayerLayout o = layer_layout(csr, layer);
  if (o.saved_total > 0 && n > 0 && !saved) return GNN_ERR_NULL;
  if (!buf16(workspace) || !buf16(saved)) return GNN_ERR_UNSUPPORTED;
  if (workspace_bytes < o.total || (o.total > 0 && !workspace))
    return GNN_ERR_WORKSPACE;
  {
    const size_t wb = (size_t)f_in * h * 4;
    const void* ins[] = {X, W_self, W_neigh, Y, dY};
    const size_t inb[] = {mat_bytes(n, f_in, layer->ld_x), wb, wb,
                          mat_bytes(n, 2 * h, layer->ld_y),
                          mat_bytes(n, 2 * h, layer->ld_y)};
    const void* outs[] = {dX, dW_self, dW_neigh, db_self, db_neigh};
    const size_t outb[] = {dX ? mat_bytes(n, f_in, layer->ld_dx) : 0, wb, wb,
                           (size_t)h * 4, (size_t)h * 4};
    for (int i = 0; i < 5; ++i)
      for (int k = 0; k < 5; ++k)
        if (ranges_overlap(outs[i], outb[i], ins[k], inb[k])) return GNN_ERR_ALIAS;
  }

  char* ws = static_cast<char*>(workspace);
  float* buf0 = reinterpret_cast<float*>(ws + o.off_buf0);
  float* buf1 = reinterpret_cast<float*>(ws + o.off_buf1);
  // weight gradients in one region; their reduction, if any, is held and
  // run by the input-gradient launch, which uses the other region
  void* wws = ws + o.off_gemm;
  const size_t wws_bytes = o.off_gemm_x - o.off_gemm;
  void* xws = ws + o.off_gemm_x;
  const size_t xws_bytes = o.off_cs - o.off_gemm_x;
  GemmFixup held;
  float* cspart = reinterpret_cast<float*>(ws + o.off_cs);

  const int32_t bf = gemm_mode(layer->flags);
  const bool dy_masked = (layer->flags & GNN_FLAG_DY_MASKED) != 0;
  // dX masked by 1[X > 0]: the next layer down's G, in the epilogue that
  // writes the final dX
  const float* dx_mask = (layer->flags & GNN_FLAG_DX_MASKED) ? X : nullptr;
  if (o.order == 2 && bf == GEMM_BF16 && !dy_masked) {
    // bf16 products: the masking pass writes G_s rounded to bf16 and G_n in
    // fp32 (the aggregation's input), the transposed aggregation writes T
    // rounded to bf16; both products read them as bf16 operands (half the
    // bytes, no conversion in the GEMM).  db_self comes from Y and dY.
    uint16_t* Gs16 = reinterpret_cast<uint16_t*>(buf0);
    uint16_t* T16 = reinterpret_cast<uint16_t*>(reinterpret_cast<char*>(buf0) + o.off_t16);
    float* G_n = buf1;
    GNN_HIP(mask_launch(n, 2 * h, h, Y, dY, layer->ld_y, Gs16, o.ld_h16, G_n, o.ld_gn, stream,
                        true));
    SpmmCall c = spmm_call(csr, true, h, G_n, o.ld_gn, reinterpret_cast<float*>(T16),
                           o.ld_h16, rn);
    c.epilogue = SPMM_STORE_BF16;
    GNN_HIP(spmm_launch(c, stream));
    const float* gs = reinterpret_cast<const float*>(Gs16);
    const float* t = reinterpret_cast<const float*>(T16);
    GemmBatch bw = dw_batch(2, n, f_in, h, X, layer->ld_x, nullptr, 0, gs, o.ld_h16, t,
                            o.ld_h16, dW_self, dW_neigh);
    bw.mode = bf;
    bw.b16 = 1;
    GNN_HIP(gemm_launch(bw, wws, wws_bytes, stream, dX ? &held : nullptr));
    if (dX) {
      GemmBatch bx = dx_batch(2, n, f_in, h, gs, o.ld_h16, t, o.ld_h16, W_self, W_neigh, dX,
                              layer->ld_dx, nullptr, 0);
      bx.mode = bf;
      bx.a16 = 1;
      bx.p[0].mask = dx_mask;
      bx.p[0].ld_mask = layer->ld_x;
      GNN_HIP(gemm_launch(bx, xws, xws_bytes, stream, nullptr, &held));
    }
    if (db_self) GNN_HIP(colsum_masked_launch(n, h, Y, dY, layer->ld_y, db_self, cspart, stream));
    if (db_neigh) GNN_HIP(colsum_launch(n, h, G_n, o.ld_gn, db_neigh, cspart, stream));
  } else if (o.order == 2) {
    // G_s and G_n: dY itself when already masked, else a masking pass
    // writes them into [G_s | T] (n x ld_g) and G_n (n x ld_gn).
    const float *Gs, *Gn;
    int64_t ld_gs, ld_gn;
    float* T;
    int64_t ld_t;
    if (dy_masked) {
      Gs = dY;
      Gn = dY + h;
      ld_gs = ld_gn = layer->ld_y;
      T = buf1;
      ld_t = o.ld_gn;
    } else {
      float* GT = buf0;
      float* G_n = buf1;
      GNN_HIP(mask_launch(n, 2 * h, h, Y, dY, layer->ld_y, GT, o.ld_g, G_n, o.ld_gn, stream));
      Gs = GT;
      ld_gs = o.ld_g;
      Gn = G_n;
      ld_gn = o.ld_gn;
      T = GT + h;
      ld_t = o.ld_g;
    }
    SpmmCall c = spmm_call(csr, true, h, Gn, ld_gn, T, ld_t, rn);
    GNN_HIP(spmm_launch(c, stream));
    GemmBatch bw = dw_batch(2, n, f_in, h, X, layer->ld_x, nullptr, 0, Gs,
                            ld_gs, T, ld_t, dW_self, dW_neigh);
    bw.mode = bf;
    GNN_HIP(gemm_launch(bw, wws, wws_bytes, stream, dX ? &held : nullptr));
    if (dX) {
      GemmBatch bx = dx_batch(2, n, f_in, h, Gs, ld_gs, T, ld_t, W_self,
                              W_neigh, dX, layer->ld_dx, nullptr, 0);
      bx.mode = bf;
      bx.p[0].mask = dx_mask;
      bx.p[0].ld_mask = layer->ld_x;
      if (bx.mode == GEMM_SPLIT && saved) {  // the pieces the forward call saved
        // (saved is NULL only for n = 0, where the product has no tiles)
        use_weight_planes(bx, W_self, saved_plane(o, saved, 0), saved_plane(o, saved, 1),
                          (int64_t)(b_planes_words(h, f_in) / 3));
      }
      GNN_HIP(gemm_launch(bx, xws, xws_bytes, stream, nullptr, &held));
    }
    if (db_self) GNN_HIP(colsum_launch(n, h, Gs, ld_gs, db_self, cspart, stream));
    if (db_neigh) GNN_HIP(colsum_launch(n, h, Gn, ld_gn, db_neigh, cspart, stream));
  } else {
    const float* G;  // [G_s | G_n]
    int64_t ld_g;
    if (dy_masked) {
      G = dY;
      ld_g = layer->ld_y;
    } else {
      float* Gm = buf0;
      GNN_HIP(mask_launch(n, 2 * h, h, Y, dY, layer->ld_y, Gm, o.ld_g, Gm + h, o.ld_g, stream));
      G = Gm;
      ld_g = o.ld_g;
    }
    float* V = buf1;  // G_n W_n^T, n x ld_v
    const float* S = static_cast<const float*>(saved);
    GemmBatch bw = dw_batch(1, n, f_in, h, X, layer->ld_x, S, o.ld_s, G, ld_g,
                            G + h, ld_g, dW_self, dW_neigh);
    bw.mode = bf;
    GNN_HIP(gemm_launch(bw, wws, wws_bytes, stream, dX ? &held : nullptr));
    if (dX) {
      GemmBatch bx = dx_batch(1, n, f_in, h, G, ld_g, G + h, ld_g, W_self,
                              W_neigh, dX, layer->ld_dx, V, o.ld_v);
      bx.mode = bf;
      if (bx.mode == GEMM_SPLIT && saved) {  // the pieces the forward call saved
        // (saved is NULL only for n = 0, where the product has no tiles)
        use_weight_planes(bx, W_self, saved_plane(o, saved, 0), saved_plane(o, saved, 1),
                          (int64_t)(b_planes_words(h, f_in) / 3));
      }
      GNN_HIP(gemm_launch(bx, xws, xws_bytes, stream, nullptr, &held));
      // dX = G_s W_s^T + A_s^T V, then the mask, in the aggregation epilogue
      SpmmCall c = spmm_call(csr, true, f_in, V, o.ld_v, dX, layer->ld_dx, rn);
      c.epilogue = SPMM_ADD;
      c.res = dX;
      c.ld_res = layer->ld_dx;
      c.mask = dx_mask;
      c.ld_mask = layer->ld_x;
      GNN_HIP(spmm_launch(c, stream));
    }
    if (db_self) GNN_HIP(colsum_launch(n, h, G, ld_g, db_self, cspart, stream));
    if (db_neigh) GNN_HIP(colsum_launch(n, h, G + h, ld_g, db_neigh, cspart, stream));
  }
  return GNN_OK;
}

gnn_status gnn_timer_enable(int32_t enable) {
  g_timer_on = enable != 0;
  return GNN_OK;
}

gnn_status gnn_timer_reset(void) {
  g_recs.clear();
  g_pool_used = 0;
  g_cur.kclass = -1;
  return GNN_OK;
}

gnn_status gnn_timer_read(int32_t kernel, double* ms, int64_t* launches,
                          double* work) {
  if (kernel < 0 || kernel >= GNN_K_COUNT) return GNN_ERR_SHAPE;
  double t = 0, wk = 0;
  int64_t c = 0;
  for (const TimerRec& r : g_recs) {
    if (r.kclass != kernel) continue;
    if (hipEventSynchronize(r.b) != hipSuccess) return GNN_ERR_HIP;
    float e = 0.f;
    if (hipEventElapsedTime(&e, r.a, r.b) != hipSuccess) return GNN_ERR_HIP;
    t += e;
    wk += r.work;
    ++c;
  }
  if (ms) *ms = t;
  if (launches) *launches = c;
  if (work) *work = wk;
  return GNN_OK;
}

}  // extern "C"
