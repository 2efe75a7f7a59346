// C-ABI of the GCN and MixHop layers (Section 2.1, Eqs. "gcn forward" and
// "mixhop forward"), built from the same aggregation, matrix-core and mask
// kernels as the GraphSAGE layer.  Their backward passes keep the A_hat
// terms of the GraphSAGE gradients (Section 5.1).
//
// GCN, Y = ReLU(A_hat X W + b), with the Section 6.1 order choice:
//   order 1:  S = A_hat X (kept);  Y = ReLU(S W + b)
//             G <- mask;  dW = S^T G;  V = G W^T;  dX = A_hat^T V
//   order 2:  P = X W;  Y = ReLU(A_hat P + b)   (bias + ReLU in the
//                                                aggregation's store)
//             G <- mask;  T = A_hat^T G;  dW = X^T T;  dX = T W^T
// MixHop, Y = ReLU(X W_0 || A_hat X W_1 || ... || A_hat^K X W_K + b):
//   S_k = A_hat S_{k-1} (S_0 = X, S_1..S_K kept);  hop k's columns of Y =
//   ReLU(S_k W_k + b_k), two hops per matrix-core launch;
//   G <- mask;  dW_k = S_k^T G_k;  dX = sum_k (A_hat^T)^k G_k W_k^T taken
//   by Horner's rule, R = G_K W_K^T, R = G_k W_k^T + A_hat^T R for
//   k = K-1 .. 0, so K aggregations (with the residual-add epilogue) and
//   K+1 products give dX.
#include <algorithm>

#include "abi.hpp"

using namespace gnnprop;

namespace {

// One product C = op(A) op(B) (+ bias, ReLU) as a one-problem batch.
GemmBatch gemm1(int trans_a, int trans_b, int32_t M, int32_t N, int32_t K,
                const float* A, int64_t lda, const float* B, int64_t ldb,
                float* C, int64_t ldc, const float* bias, int relu,
                uint32_t flags) {
  GemmBatch b;
  memset(&b, 0, sizeof(b));
  b.nprob = 1;
  b.trans_a = trans_a;
  b.trans_b = trans_b;
  b.mode = gemm_mode(flags);
  GemmProblem& p = b.p[0];
  p.nseg = 1;
  p.seg[0] = {A, B, lda, ldb, K};
  p.M = M;
  p.N = N;
  p.C = C;
  p.ldc = ldc;
  p.bias = bias;
  p.relu = relu;
  return b;
}

// Two products of the same M and K in one launch.
GemmBatch gemm2(const GemmBatch& a, const GemmBatch& b) {
  GemmBatch c = a;
  c.nprob = 2;
  c.p[1] = b.p[0];
  return c;
}

gnn_status check_variant_layer(const gnn_layer* L, int64_t width_y) {
  if (!L) return GNN_ERR_NULL;
  if (L->f_in <= 0 || L->h <= 0) return GNN_ERR_SHAPE;
  if (L->ld_x < L->f_in || L->ld_y < width_y) return GNN_ERR_SHAPE;
  if (L->order < 0 || L->order > 2) return GNN_ERR_SHAPE;
  if ((L->flags & ~GEMM_FLAGS) || !gemm_flags_ok(L->flags)) return GNN_ERR_UNSUPPORTED;
  return GNN_OK;
}

size_t gemm_ws(const GemmBatch& b) { return gemm_workspace_bytes(b); }

// ---------------------------------------------------------------- GCN

struct GcnLayout {
  int order;
  int64_t ld_s, ld_h, ld_b;
  // GEMM workspace: [off_gemm, off_gemm_x) the weight gradient's partial
  // tiles, summed by the input-gradient launch; [off_gemm_x, off_cs) the rest
  size_t off_a, off_b, off_gemm, off_gemm_x, off_cs, total;
};

GcnLayout gcn_layout(const gnn_csr* csr, const gnn_layer* L) {
  GcnLayout o;
  const int32_t n = csr->n, f_in = L->f_in, h = L->h;
  o.order = L->order ? L->order : gnn_choose_order(f_in, h);
  o.ld_s = round_up(f_in, 4);
  o.ld_h = round_up(h, 4);
  o.ld_b = std::max(o.ld_h, o.ld_s);
  const size_t a = (size_t)n * o.ld_h * 4;  // P or G
  const size_t b = (size_t)n * o.ld_b * 4;  // T or V
  const size_t gw = gemm_ws(gemm1(1, 0, f_in, h, n, 0, f_in, 0, h, 0, h, 0, 0, L->flags));
  const size_t g =
      std::max(gemm_ws(gemm1(0, 0, n, h, f_in, 0, f_in, 0, h, 0, h, 0, 0, L->flags)),
               gemm_ws(gemm1(0, 1, n, f_in, h, 0, h, 0, h, 0, f_in, 0, 0, L->flags)));
  o.off_a = 0;
  o.off_b = round_up(a, 256);
  o.off_gemm = o.off_b + round_up(b, 256);
  o.off_gemm_x = o.off_gemm + round_up(gw, 256);
  o.off_cs = o.off_gemm_x + round_up(g, 256);
  o.total = o.off_cs + colsum_partials_bytes(n, h);
  return o;
}

// ------------------------------------------------------------- MixHop

struct MixLayout {
  int64_t ld_s, ld_g, ld_r;
  // GEMM workspace: the weight-gradient launches' partial tiles alternate
  // between [off_gemm, off_gemm + gw) and the gw bytes after it (each
  // launch sums its predecessor's, the first input-gradient launch the
  // last's); [off_gemm_x, off_cs) serves the other launches
  size_t saved, off_g, off_r0, off_r1, off_gemm, gw, off_gemm_x, off_cs, total;
};

MixLayout mix_layout(const gnn_csr* csr, const gnn_layer* L, int32_t K) {
  MixLayout o;
  const int32_t n = csr->n, f_in = L->f_in, h = L->h;
  const int32_t wy = (K + 1) * h;
  o.ld_s = round_up(f_in, 4);
  o.ld_g = round_up(wy, 4);
  o.ld_r = round_up(f_in, 4);
  o.saved = (size_t)K * n * o.ld_s * 4;
  size_t g = 0, gw = 0;
  const GemmBatch f = gemm1(0, 0, n, h, f_in, 0, f_in, 0, wy, 0, wy, 0, 1, L->flags);
  const GemmBatch w = gemm1(1, 0, f_in, h, n, 0, f_in, 0, wy, 0, wy, 0, 0, L->flags);
  // hops go two per launch, the last one alone when K + 1 is odd; the work
  // split (and so the workspace) differs between the two shapes
  g = std::max(g, gemm_ws(f));
  gw = std::max(gw, gemm_ws(w));
  if (K > 0) {
    g = std::max(g, gemm_ws(gemm2(f, f)));
    gw = std::max(gw, gemm_ws(gemm2(w, w)));
  }
  g = std::max(g, gemm_ws(gemm1(0, 1, n, f_in, h, 0, wy, 0, wy, 0, f_in, 0, 0, L->flags)));
  o.gw = round_up(gw, 256);
  o.off_g = 0;
  o.off_r0 = round_up((size_t)n * o.ld_g * 4, 256);
  o.off_r1 = o.off_r0 + round_up((size_t)n * o.ld_r * 4, 256);
  o.off_gemm = o.off_r1 + round_up((size_t)n * o.ld_r * 4, 256);
  o.off_gemm_x = o.off_gemm + (K >= 2 ? 2 : 1) * o.gw;  // K >= 2: several dW launches
  o.off_cs = o.off_gemm_x + round_up(g, 256);
  o.total = o.off_cs + colsum_partials_bytes(n, wy);
  return o;
}

}  // namespace

extern "C" {

size_t gnn_gcn_saved_bytes(const gnn_csr* csr, const gnn_layer* layer) {
  if (!csr || check_variant_layer(layer, layer ? layer->h : 0) != GNN_OK) return 0;
  const GcnLayout o = gcn_layout(csr, layer);
  return o.order == 1 ? (size_t)csr->n * o.ld_s * 4 : 0;
}

size_t gnn_gcn_workspace_bytes(const gnn_csr* csr, const gnn_layer* layer) {
  if (!csr || check_variant_layer(layer, layer ? layer->h : 0) != GNN_OK) return 0;
  return gcn_layout(csr, layer).total;
}

gnn_status gnn_gcn_fwd(const gnn_csr* csr, const gnn_layer* layer,
                       const float* X, const float* W, const float* b,
                       float* Y, void* saved, void* workspace,
                       size_t workspace_bytes, hipStream_t stream) {
  gnn_status st = check_csr(csr, true, false);
  if (st != GNN_OK) return st;
  if ((st = check_variant_layer(layer, layer ? layer->h : 0)) != GNN_OK) return st;
  const int32_t n = csr->n, f_in = layer->f_in, h = layer->h;
  if (!W) return GNN_ERR_NULL;
  if (n > 0 && (!X || !Y || !csr->plan)) return GNN_ERR_NULL;
  const GcnLayout o = gcn_layout(csr, layer);
  if (o.order == 1 && n > 0 && !saved) return GNN_ERR_NULL;
  if (!buf16(workspace) || !buf16(saved)) return GNN_ERR_UNSUPPORTED;
  if (workspace_bytes < o.total || (o.total > 0 && !workspace))
    return GNN_ERR_WORKSPACE;
  if (n == 0) return GNN_OK;
  const size_t yb = mat_bytes(n, h, layer->ld_y);
  if (ranges_overlap(Y, yb, X, mat_bytes(n, f_in, layer->ld_x)) ||
      ranges_overlap(Y, yb, W, (size_t)f_in * h * 4))
    return GNN_ERR_ALIAS;
  char* ws = static_cast<char*>(workspace);
  void* gws = ws + o.off_gemm;
  const size_t gws_bytes = o.off_cs - o.off_gemm;
  if (o.order == 1) {
    float* S = static_cast<float*>(saved);
    GNN_HIP(spmm_launch(spmm_call(csr, false, f_in, X, layer->ld_x, S, o.ld_s), stream));
    GNN_HIP(gemm_launch(gemm1(0, 0, n, h, f_in, S, o.ld_s, W, h, Y, layer->ld_y, b, 1,
                              layer->flags), gws, gws_bytes, stream));
  } else {
    float* P = reinterpret_cast<float*>(ws + o.off_a);
    GNN_HIP(gemm_launch(gemm1(0, 0, n, h, f_in, X, layer->ld_x, W, h, P, o.ld_h, nullptr,
                              0, layer->flags), gws, gws_bytes, stream));
    SpmmCall c = spmm_call(csr, false, h, P, o.ld_h, Y, layer->ld_y);
    c.epilogue = SPMM_BIAS_RELU;
    c.bias = b;
    GNN_HIP(spmm_launch(c, stream));
  }
  return GNN_OK;
}

gnn_status gnn_gcn_bwd(const gnn_csr* csr, const gnn_layer* layer,
                       const float* X, const float* W, const float* Y,
                       const float* dY, const void* saved, float* dX,
                       float* dW, float* db, void* workspace,
                       size_t workspace_bytes, hipStream_t stream) {
  gnn_status st = check_csr(csr, true, true);
  if (st != GNN_OK) return st;
  if ((st = check_variant_layer(layer, layer ? layer->h : 0)) != GNN_OK) return st;
  const int32_t n = csr->n, f_in = layer->f_in, h = layer->h;
  if (!W || !dW) return GNN_ERR_NULL;
  if (n > 0 && (!X || !Y || !dY || !csr->plan)) return GNN_ERR_NULL;
  if (dX && layer->ld_dx < f_in) return GNN_ERR_SHAPE;
  const GcnLayout o = gcn_layout(csr, layer);
  if (o.order == 1 && n > 0 && !saved) return GNN_ERR_NULL;
  if (!buf16(workspace) || !buf16(saved)) return GNN_ERR_UNSUPPORTED;
  if (workspace_bytes < o.total || (o.total > 0 && !workspace))
    return GNN_ERR_WORKSPACE;
  {
    const void* ins[] = {X, W, Y, dY};
    const size_t inb[] = {mat_bytes(n, f_in, layer->ld_x), (size_t)f_in * h * 4,
                          mat_bytes(n, h, layer->ld_y), mat_bytes(n, h, layer->ld_y)};
    const void* outs[] = {dX, dW, db};
    const size_t outb[] = {dX ? mat_bytes(n, f_in, layer->ld_dx) : 0,
                           (size_t)f_in * h * 4, (size_t)h * 4};
    for (int i = 0; i < 3; ++i)
      for (int k = 0; k < 4; ++k)
        if (ranges_overlap(outs[i], outb[i], ins[k], inb[k])) return GNN_ERR_ALIAS;
  }
  char* ws = static_cast<char*>(workspace);
  float* G = reinterpret_cast<float*>(ws + o.off_a);
  float* B = reinterpret_cast<float*>(ws + o.off_b);
  // the weight gradient's reduction, if any, is held for the input-gradient
  // launch, which takes the other workspace region
  void* wws = ws + o.off_gemm;
  const size_t wws_bytes = o.off_gemm_x - o.off_gemm;
  void* xws = ws + o.off_gemm_x;
  const size_t xws_bytes = o.off_cs - o.off_gemm_x;
  GemmFixup held;
  float* cspart = reinterpret_cast<float*>(ws + o.off_cs);
  GNN_HIP(mask_launch(n, h, h, Y, dY, layer->ld_y, G, o.ld_h, nullptr, 0, stream));
  if (o.order == 1) {
    const float* S = static_cast<const float*>(saved);
    GNN_HIP(gemm_launch(gemm1(1, 0, f_in, h, n, S, o.ld_s, G, o.ld_h, dW, h, nullptr, 0,
                              layer->flags), wws, wws_bytes, stream, dX ? &held : nullptr));
    if (dX) {
      float* V = B;
      GNN_HIP(gemm_launch(gemm1(0, 1, n, f_in, h, G, o.ld_h, W, h, V, o.ld_b, nullptr, 0,
                                layer->flags), xws, xws_bytes, stream, nullptr, &held));
      GNN_HIP(spmm_launch(spmm_call(csr, true, f_in, V, o.ld_b, dX, layer->ld_dx), stream));
    }
  } else {
    float* T = B;
    GNN_HIP(spmm_launch(spmm_call(csr, true, h, G, o.ld_h, T, o.ld_b), stream));
    GNN_HIP(gemm_launch(gemm1(1, 0, f_in, h, n, X, layer->ld_x, T, o.ld_b, dW, h, nullptr,
                              0, layer->flags), wws, wws_bytes, stream, dX ? &held : nullptr));
    if (dX)
      GNN_HIP(gemm_launch(gemm1(0, 1, n, f_in, h, T, o.ld_b, W, h, dX, layer->ld_dx,
                                nullptr, 0, layer->flags), xws, xws_bytes, stream, nullptr,
                          &held));
  }
  if (db) GNN_HIP(colsum_launch(n, h, G, o.ld_h, db, cspart, stream));
  return GNN_OK;
}

size_t gnn_mixhop_saved_bytes(const gnn_csr* csr, const gnn_layer* layer,
                              int32_t K) {
  if (!csr || K < 0 || !layer) return 0;
  if (check_variant_layer(layer, (int64_t)(K + 1) * layer->h) != GNN_OK) return 0;
  return mix_layout(csr, layer, K).saved;
}

size_t gnn_mixhop_workspace_bytes(const gnn_csr* csr, const gnn_layer* layer,
                                  int32_t K) {
  if (!csr || K < 0 || !layer) return 0;
  if (check_variant_layer(layer, (int64_t)(K + 1) * layer->h) != GNN_OK) return 0;
  return mix_layout(csr, layer, K).total;
}

gnn_status gnn_mixhop_fwd(const gnn_csr* csr, const gnn_layer* layer,
                          int32_t K, const float* X, const float* W,
                          const float* b, float* Y, void* saved,
                          void* workspace, size_t workspace_bytes,
                          hipStream_t stream) {
  gnn_status st = check_csr(csr, true, false);
  if (st != GNN_OK) return st;
  if (K < 0) return GNN_ERR_SHAPE;
  if (!layer) return GNN_ERR_NULL;
  if ((st = check_variant_layer(layer, (int64_t)(K + 1) * layer->h)) != GNN_OK) return st;
  if (layer->order == 2) return GNN_ERR_UNSUPPORTED;
  const int32_t n = csr->n, f_in = layer->f_in, h = layer->h, wy = (K + 1) * h;
  if (!W) return GNN_ERR_NULL;
  if (n > 0 && (!X || !Y || !csr->plan || (K > 0 && !saved))) return GNN_ERR_NULL;
  const MixLayout o = mix_layout(csr, layer, K);
  if (!buf16(workspace) || !buf16(saved)) return GNN_ERR_UNSUPPORTED;
  if (workspace_bytes < o.total || (o.total > 0 && !workspace))
    return GNN_ERR_WORKSPACE;
  if (n == 0) return GNN_OK;
  const size_t yb = mat_bytes(n, wy, layer->ld_y);
  if (ranges_overlap(Y, yb, X, mat_bytes(n, f_in, layer->ld_x)) ||
      ranges_overlap(Y, yb, W, (size_t)f_in * wy * 4))
    return GNN_ERR_ALIAS;
  char* ws = static_cast<char*>(workspace);
  void* gws = ws + o.off_gemm;
  const size_t gws_bytes = o.off_cs - o.off_gemm;
  float* Sv = static_cast<float*>(saved);
  auto S = [&](int k) -> const float* {
    return k == 0 ? X : Sv + (size_t)(k - 1) * n * o.ld_s;
  };
  auto ldS = [&](int k) { return k == 0 ? layer->ld_x : o.ld_s; };
  for (int k = 1; k <= K; ++k)
    GNN_HIP(spmm_launch(spmm_call(csr, false, f_in, S(k - 1), ldS(k - 1),
                                  Sv + (size_t)(k - 1) * n * o.ld_s, o.ld_s), stream));
  auto hop = [&](int k) {
    return gemm1(0, 0, n, h, f_in, S(k), ldS(k), W + (size_t)k * h, wy,
                 Y + (size_t)k * h, layer->ld_y, b ? b + (size_t)k * h : nullptr, 1,
                 layer->flags);
  };
  for (int k = 0; k <= K; k += 2) {
    const GemmBatch bt = k + 1 <= K ? gemm2(hop(k), hop(k + 1)) : hop(k);
    GNN_HIP(gemm_launch(bt, gws, gws_bytes, stream));
  }
  return GNN_OK;
}

gnn_status gnn_mixhop_bwd(const gnn_csr* csr, const gnn_layer* layer,
                          int32_t K, const float* X, const float* W,
                          const float* Y, const float* dY, const void* saved,
                          float* dX, float* dW, float* db, void* workspace,
                          size_t workspace_bytes, hipStream_t stream) {
  gnn_status st = check_csr(csr, true, true);
  if (st != GNN_OK) return st;
  if (K < 0) return GNN_ERR_SHAPE;
  if (!layer) return GNN_ERR_NULL;
  if ((st = check_variant_layer(layer, (int64_t)(K + 1) * layer->h)) != GNN_OK) return st;
  if (layer->order == 2) return GNN_ERR_UNSUPPORTED;
  const int32_t n = csr->n, f_in = layer->f_in, h = layer->h, wy = (K + 1) * h;
  if (!W || !dW) return GNN_ERR_NULL;
  if (n > 0 && (!X || !Y || !dY || !csr->plan || (K > 0 && !saved))) return GNN_ERR_NULL;
  if (dX && layer->ld_dx < f_in) return GNN_ERR_SHAPE;
  const MixLayout o = mix_layout(csr, layer, K);
  if (!buf16(workspace) || !buf16(saved)) return GNN_ERR_UNSUPPORTED;
  if (workspace_bytes < o.total || (o.total > 0 && !workspace))
    return GNN_ERR_WORKSPACE;
  {
    const void* ins[] = {X, W, Y, dY};
    const size_t inb[] = {mat_bytes(n, f_in, layer->ld_x), (size_t)f_in * wy * 4,
                          mat_bytes(n, wy, layer->ld_y), mat_bytes(n, wy, layer->ld_y)};
    const void* outs[] = {dX, dW, db};
    const size_t outb[] = {dX ? mat_bytes(n, f_in, layer->ld_dx) : 0,
                           (size_t)f_in * wy * 4, (size_t)wy * 4};
    for (int i = 0; i < 3; ++i)
      for (int k = 0; k < 4; ++k)
        if (ranges_overlap(outs[i], outb[i], ins[k], inb[k])) return GNN_ERR_ALIAS;
  }
  char* ws = static_cast<char*>(workspace);
  float* G = reinterpret_cast<float*>(ws + o.off_g);
  float* R[2] = {reinterpret_cast<float*>(ws + o.off_r0),
                 reinterpret_cast<float*>(ws + o.off_r1)};
  void* xws = ws + o.off_gemm_x;
  const size_t xws_bytes = o.off_cs - o.off_gemm_x;
  float* cspart = reinterpret_cast<float*>(ws + o.off_cs);
  const float* Sv = static_cast<const float*>(saved);
  auto S = [&](int k) -> const float* {
    return k == 0 ? X : Sv + (size_t)(k - 1) * n * o.ld_s;
  };
  auto ldS = [&](int k) { return k == 0 ? layer->ld_x : o.ld_s; };
  GNN_HIP(mask_launch(n, wy, wy, Y, dY, layer->ld_y, G, o.ld_g, nullptr, 0, stream));
  // dW_k = S_k^T G_k, two hops per launch; each launch's reduction is held
  // and summed by extra blocks of the next GEMM launch (the partial tiles
  // alternate between two regions)
  auto dw = [&](int k) {
    return gemm1(1, 0, f_in, h, n, S(k), ldS(k), G + (size_t)k * h, o.ld_g,
                 dW + (size_t)k * h, wy, nullptr, 0, layer->flags);
  };
  GemmFixup held[2];
  const GemmFixup* pend = nullptr;
  for (int k = 0, i = 0; k <= K; k += 2, ++i) {
    const GemmBatch bt = k + 1 <= K ? gemm2(dw(k), dw(k + 1)) : dw(k);
    GNN_HIP(gemm_launch(bt, ws + o.off_gemm + (i & 1) * o.gw, o.gw, stream, &held[i & 1],
                        pend));
    pend = &held[i & 1];
  }
  if (!dX && pend) GNN_HIP(gemm_flush(*pend, stream));
  if (db) GNN_HIP(colsum_launch(n, wy, G, o.ld_g, db, cspart, stream));
  if (dX) {
    // Horner: R = G_K W_K^T;  R = G_k W_k^T + A_hat^T R for k = K-1 .. 0,
    // the last step written into dX.
    auto vk = [&](int k, float* out, int64_t ld_out) {
      return gemm1(0, 1, n, f_in, h, G + (size_t)k * h, o.ld_g, W + (size_t)k * h, wy,
                   out, ld_out, nullptr, 0, layer->flags);
    };
    int cur = 0;
    float* r = K == 0 ? dX : R[cur];
    int64_t ld_r = K == 0 ? layer->ld_dx : o.ld_r;
    GNN_HIP(gemm_launch(vk(K, r, ld_r), xws, xws_bytes, stream, nullptr, pend));
    for (int k = K - 1; k >= 0; --k) {
      float* nx = k == 0 ? dX : R[cur ^ 1];
      const int64_t ld_nx = k == 0 ? layer->ld_dx : o.ld_r;
      GNN_HIP(gemm_launch(vk(k, nx, ld_nx), xws, xws_bytes, stream));
      SpmmCall c = spmm_call(csr, true, f_in, r, ld_r, nx, ld_nx);
      c.epilogue = SPMM_ADD;
      c.res = nx;
      c.ld_res = ld_nx;
      GNN_HIP(spmm_launch(c, stream));
      cur ^= 1;
      r = nx;
      ld_r = ld_nx;
    }
  }
  return GNN_OK;
}

}  // extern "C"
