// C-ABI of the GAT layer (Section 2.1, Eqs. "gat forward" and "gat
// attention") on the aggregation and matrix-core kernels, plus the three
// kernels the attention adds: per-node scores, per-entry attention values,
// and the per-entry dot products of the backward pass (an SDDMM).
//
// Forward, with a = [a1; a2] (2h) and slope alpha:
//   P = X W                               (matrix cores; kept)
//   s_u = a1 . P_u,  t_u = a2 . P_u       (one wavefront per row; kept)
//   att_j = LeakyReLU(s_u + t_v)          (entry j = (u, v); kept)
//   Y = ReLU(A_att P)                     (aggregation with att as values)
// since a . (P_u || P_v) = s_u + t_v, the attention costs O(nnz) once the
// scores are known.  Backward (chain rule):
//   G = dY * 1[Y > 0]
//   dz_j = (G_u . P_v) * (att_j > 0 ? 1 : alpha)        (SDDMM)
//   ds_u = sum over row u of dz,  dt_v = sum over column v of dz (row sums
//     of the transposed values, Algorithm 6's permutation)
//   dP = A_att^T G + ds a1^T + dt a2^T   (aggregation on the transposed
//                                         attention, then a rank-2 update)
//   da1 = P^T ds, da2 = P^T dt (weighted column sums, fixed order),
//   dW = X^T dP,  dX = dP W^T                             (matrix cores)
#include <algorithm>

#include "abi.hpp"

using namespace gnnprop;

namespace {

__device__ inline float wave_sum(float v) {
#pragma unroll
  for (int d = 32; d > 0; d >>= 1) v += __shfl_xor(v, d, 64);
  return v;
}

// s_u = a1 . P_u and t_u = a2 . P_u, one wavefront per row.
__global__ __launch_bounds__(256) void gat_scores_kernel(
    int32_t n, int32_t h, const float* __restrict__ P, int64_t ld_p,
    const float* __restrict__ a, float* __restrict__ s, float* __restrict__ t) {
  const int32_t u = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (u >= n) return;
  const float* p = P + (int64_t)u * ld_p;
  float x = 0.f, y = 0.f;
  for (int32_t c = lane; c < h; c += 64) {
    const float v = p[c];
    x += a[c] * v;
    y += a[h + c] * v;
  }
  x = wave_sum(x);
  y = wave_sum(y);
  if (lane == 0) {
    s[u] = x;
    t[u] = y;
  }
}

// att_j = LeakyReLU(s[row_j] + t[col_j]).
__global__ __launch_bounds__(256) void gat_att_kernel(
    int64_t nnz, const int32_t* __restrict__ erow, const int32_t* __restrict__ indices,
    const float* __restrict__ s, const float* __restrict__ t, float alpha,
    float* __restrict__ att) {
  const int64_t j = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (j >= nnz) return;
  const float z = s[erow[j]] + t[indices[j]];
  att[j] = z > 0.f ? z : alpha * z;
}

// dz_j = (G_u . P_v) * (att_j > 0 ? 1 : alpha) for entry j = (u, v): a
// group of 16 lanes per entry, each lane a float4 column strip; entries in
// CSR order, so consecutive groups share G_u in the cache and gather P_v.
template <bool VEC>
__global__ __launch_bounds__(256) void gat_sddmm_kernel(
    int64_t nnz, int32_t h, const int32_t* __restrict__ erow,
    const int32_t* __restrict__ indices, const float* __restrict__ G, int64_t ld_g,
    const float* __restrict__ P, int64_t ld_p, const float* __restrict__ att,
    float alpha, float* __restrict__ dz) {
  const int gl = threadIdx.x & 15;
  for (int64_t j = (int64_t)blockIdx.x * 16 + (threadIdx.x >> 4); j < nnz;
       j += (int64_t)gridDim.x * 16) {
    const float* g = G + (int64_t)erow[j] * ld_g;
    const float* p = P + (int64_t)indices[j] * ld_p;
    float acc = 0.f;
    if (VEC) {
      for (int32_t c = 4 * gl; c < h; c += 64) {
        const float4 x = *reinterpret_cast<const float4*>(g + c);
        const float4 y = *reinterpret_cast<const float4*>(p + c);
        acc += x.x * y.x + x.y * y.y + x.z * y.z + x.w * y.w;
      }
    } else {
      for (int32_t c = gl; c < h; c += 16) acc += g[c] * p[c];
    }
#pragma unroll
    for (int d = 8; d > 0; d >>= 1) acc += __shfl_xor(acc, d, 16);
    if (gl == 0) dz[j] = acc * (att[j] > 0.f ? 1.f : alpha);
  }
}

// ds_u = sum over row u of dz, dt_u = sum over row u of dz_t (the values of
// the transposed pattern), one wavefront per row, in entry order.
__global__ __launch_bounds__(256) void gat_rowsums_kernel(
    int32_t n, const int32_t* __restrict__ indptr, const float* __restrict__ dz,
    const float* __restrict__ dz_t, float* __restrict__ ds, float* __restrict__ dt) {
  const int32_t u = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (u >= n) return;
  float x = 0.f, y = 0.f;
  for (int32_t j = indptr[u] + lane; j < indptr[u + 1]; j += 64) {
    x += dz[j];
    y += dz_t[j];
  }
  x = wave_sum(x);
  y = wave_sum(y);
  if (lane == 0) {
    ds[u] = x;
    dt[u] = y;
  }
}

// dP[u, c] += ds_u a1[c] + dt_u a2[c], one thread per element.
__global__ __launch_bounds__(256) void gat_rank2_kernel(
    int32_t n, int32_t h, const float* __restrict__ ds, const float* __restrict__ dt,
    const float* __restrict__ a, float* __restrict__ dP, int64_t ld) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= (int64_t)n * h) return;
  const int32_t u = (int32_t)(i / h), c = (int32_t)(i % h);
  dP[(int64_t)u * ld + c] += ds[u] * a[c] + dt[u] * a[h + c];
}

GemmBatch gemm1(int ta, int tb, int32_t M, int32_t N, int32_t K, const float* A,
                int64_t lda, const float* B, int64_t ldb, float* C, int64_t ldc,
                int relu, uint32_t flags) {
  GemmBatch b;
  memset(&b, 0, sizeof(b));
  b.nprob = 1;
  b.trans_a = ta;
  b.trans_b = tb;
  b.mode = gemm_mode(flags);
  b.p[0].nseg = 1;
  b.p[0].seg[0] = {A, B, lda, ldb, K};
  b.p[0].M = M;
  b.p[0].N = N;
  b.p[0].C = C;
  b.p[0].ldc = ldc;
  b.p[0].relu = relu;
  return b;
}

gnn_status check_gat(const gnn_csr* csr, const gnn_layer* L, float alpha) {
  gnn_status st = check_csr(csr, false, false);
  if (st != GNN_OK) return st;
  if (!L) return GNN_ERR_NULL;
  if (L->f_in <= 0 || L->h <= 0) return GNN_ERR_SHAPE;
  if (L->ld_x < L->f_in || L->ld_y < L->h) return GNN_ERR_SHAPE;
  if ((L->flags & ~GEMM_FLAGS) || !gemm_flags_ok(L->flags)) return GNN_ERR_UNSUPPORTED;
  if (!(alpha >= 0.f && alpha <= 1.f)) return GNN_ERR_SHAPE;
  return GNN_OK;
}

// saved: P (n x ld_h), s, t (n), att (nnz).
// workspace: G (n x ld_h), dP (n x ld_h), dz, dz_t, att_t (nnz), [ds; dt]
// (2 x ld_n), column-sum partials, GEMM partials.
struct GatLayout {
  int64_t ld_h, ld_n;
  size_t s_p, s_s, s_t, s_att, saved;
  // GEMM workspace: [w_gemm, w_gemm_x) the weight gradient's partial tiles,
  // summed by the input-gradient launch; [w_gemm_x, total) the rest
  size_t w_g, w_dp, w_dz, w_dzt, w_att_t, w_dsdt, w_cs, w_gemm, w_gemm_x, total;
};

GatLayout gat_layout(const gnn_csr* csr, const gnn_layer* L) {
  GatLayout o;
  const int32_t n = csr->n, f_in = L->f_in, h = L->h;
  const int64_t nnz = csr->nnz;
  o.ld_h = round_up(h, 4);
  o.ld_n = round_up(std::max(n, 1), 4);
  const size_t nh = round_up((size_t)n * o.ld_h * 4, 256);
  const size_t nb = round_up((size_t)std::max(n, 1) * 4, 256);
  const size_t eb = round_up((size_t)std::max<int64_t>(nnz, 1) * 4, 256);
  o.s_p = 0;
  o.s_s = nh;
  o.s_t = o.s_s + nb;
  o.s_att = o.s_t + nb;
  o.saved = o.s_att + eb;
  const size_t gw =
      gemm_workspace_bytes(gemm1(1, 0, f_in, h, n, 0, f_in, 0, h, 0, h, 0, L->flags));
  const size_t g = std::max(
      gemm_workspace_bytes(gemm1(0, 0, n, h, f_in, 0, f_in, 0, h, 0, h, 0, L->flags)),
      gemm_workspace_bytes(gemm1(0, 1, n, f_in, h, 0, h, 0, h, 0, f_in, 0, L->flags)));
  o.w_g = 0;
  o.w_dp = nh;
  o.w_dz = o.w_dp + nh;
  o.w_dzt = o.w_dz + eb;
  o.w_att_t = o.w_dzt + eb;
  o.w_dsdt = o.w_att_t + eb;
  o.w_cs = o.w_dsdt + round_up((size_t)2 * o.ld_n * 4, 256);
  o.w_gemm = o.w_cs + colsum_partials_bytes(n, h, 2);
  o.w_gemm_x = o.w_gemm + round_up(gw, 256);
  o.total = o.w_gemm_x + round_up(g, 256);
  return o;
}

const int32_t* plan_erow(const gnn_csr* csr) {
  const PlanDims d = plan_dims(csr->n, csr->nnz);
  return reinterpret_cast<const int32_t*>(static_cast<const char*>(csr->plan) +
                                          d.erow_offset);
}

}  // namespace

extern "C" {

size_t gnn_gat_saved_bytes(const gnn_csr* csr, const gnn_layer* layer) {
  if (check_gat(csr, layer, 0.f) != GNN_OK) return 0;
  return gat_layout(csr, layer).saved;
}

size_t gnn_gat_workspace_bytes(const gnn_csr* csr, const gnn_layer* layer) {
  if (check_gat(csr, layer, 0.f) != GNN_OK) return 0;
  return gat_layout(csr, layer).total;
}

gnn_status gnn_gat_fwd(const gnn_csr* csr, const gnn_layer* layer, const float* X,
                       const float* W, const float* a, float alpha, float* Y,
                       float* att_out, void* saved, void* workspace,
                       size_t workspace_bytes, hipStream_t stream) {
  gnn_status st = check_gat(csr, layer, alpha);
  if (st != GNN_OK) return st;
  const int32_t n = csr->n, f_in = layer->f_in, h = layer->h;
  const int64_t nnz = csr->nnz;
  if (!W || !a) return GNN_ERR_NULL;
  if (n > 0 && (!X || !Y || !saved || !csr->plan)) return GNN_ERR_NULL;
  const GatLayout o = gat_layout(csr, layer);
  if (!buf16(workspace) || !buf16(saved)) return GNN_ERR_UNSUPPORTED;
  if (workspace_bytes < o.total || !workspace) return GNN_ERR_WORKSPACE;
  {
    const void* ins[] = {X, W, a};
    const size_t inb[] = {mat_bytes(n, f_in, layer->ld_x), (size_t)f_in * h * 4,
                          (size_t)2 * h * 4};
    const void* outs[] = {Y, att_out, saved, workspace};
    const size_t outb[] = {mat_bytes(n, h, layer->ld_y), att_out ? (size_t)nnz * 4 : 0,
                           o.saved, o.total};
    for (int i = 0; i < 4; ++i) {
      for (int k = 0; k < 3; ++k)
        if (ranges_overlap(outs[i], outb[i], ins[k], inb[k])) return GNN_ERR_ALIAS;
      for (int k = 0; k < i; ++k)
        if (ranges_overlap(outs[i], outb[i], outs[k], outb[k])) return GNN_ERR_ALIAS;
    }
  }
  if (n == 0) return GNN_OK;
  char* sv = static_cast<char*>(saved);
  float* P = reinterpret_cast<float*>(sv + o.s_p);
  float* s = reinterpret_cast<float*>(sv + o.s_s);
  float* t = reinterpret_cast<float*>(sv + o.s_t);
  float* att = reinterpret_cast<float*>(sv + o.s_att);
  char* ws = static_cast<char*>(workspace);
  GNN_HIP(gemm_launch(gemm1(0, 0, n, h, f_in, X, layer->ld_x, W, h, P, o.ld_h, 0,
                            layer->flags),
                      ws + o.w_gemm, o.total - o.w_gemm, stream));
  gat_scores_kernel<<<(unsigned)ceil_div(n, 4), 256, 0, stream>>>(n, h, P, o.ld_h, a, s, t);
  if (nnz > 0)
    gat_att_kernel<<<(unsigned)ceil_div(nnz, 256), 256, 0, stream>>>(
        nnz, plan_erow(csr), csr->indices, s, t, alpha, att);
  GNN_HIP(hipGetLastError());
  SpmmCall c = spmm_call(csr, false, h, P, o.ld_h, Y, layer->ld_y);
  c.vals = att;
  c.epilogue = SPMM_BIAS_RELU;
  GNN_HIP(spmm_launch(c, stream));
  if (att_out && nnz > 0)
    GNN_HIP(hipMemcpyAsync(att_out, att, (size_t)nnz * 4, hipMemcpyDeviceToDevice, stream));
  return GNN_OK;
}

gnn_status gnn_gat_bwd(const gnn_csr* csr, const gnn_layer* layer, const float* X,
                       const float* W, const float* a, float alpha, const float* Y,
                       const float* dY, const void* saved, float* dX, float* dW,
                       float* da, void* workspace, size_t workspace_bytes,
                       hipStream_t stream) {
  gnn_status st = check_gat(csr, layer, alpha);
  if (st != GNN_OK) return st;
  const int32_t n = csr->n, f_in = layer->f_in, h = layer->h;
  const int64_t nnz = csr->nnz;
  if (!W || !a || !dW || !da) return GNN_ERR_NULL;
  if (n > 0 && (!X || !Y || !dY || !saved || !csr->plan)) return GNN_ERR_NULL;
  if (dX && layer->ld_dx < f_in) return GNN_ERR_SHAPE;
  const GatLayout o = gat_layout(csr, layer);
  if (!buf16(workspace) || !buf16(saved)) return GNN_ERR_UNSUPPORTED;
  if (workspace_bytes < o.total || !workspace) return GNN_ERR_WORKSPACE;
  {
    const size_t wb = (size_t)f_in * h * 4;
    const void* ins[] = {X, W, a, Y, dY, saved};
    const size_t inb[] = {mat_bytes(n, f_in, layer->ld_x), wb, (size_t)2 * h * 4,
                          mat_bytes(n, h, layer->ld_y), mat_bytes(n, h, layer->ld_y),
                          o.saved};
    const void* outs[] = {dX, dW, da, workspace};
    const size_t outb[] = {dX ? mat_bytes(n, f_in, layer->ld_dx) : 0, wb,
                           (size_t)2 * h * 4, o.total};
    for (int i = 0; i < 4; ++i) {
      for (int k = 0; k < 6; ++k)
        if (ranges_overlap(outs[i], outb[i], ins[k], inb[k])) return GNN_ERR_ALIAS;
      for (int k = 0; k < i; ++k)
        if (ranges_overlap(outs[i], outb[i], outs[k], outb[k])) return GNN_ERR_ALIAS;
    }
  }
  char* ws = static_cast<char*>(workspace);
  void* gws = ws + o.w_gemm;
  const size_t gws_bytes = o.total - o.w_gemm;
  if (n == 0) {  // no rows: zero gradients through empty products
    GNN_HIP(gemm_launch(gemm1(1, 0, f_in, h, 0, X, layer->ld_x, dY, layer->ld_y, dW, h, 0,
                              layer->flags), gws, gws_bytes, stream));
    float* cspart = reinterpret_cast<float*>(ws + o.w_cs);
    GNN_HIP(colsum_launch(0, h, dY, h, da, cspart, stream));
    GNN_HIP(colsum_launch(0, h, dY, h, da + h, cspart, stream));
    return GNN_OK;
  }
  const char* sv = static_cast<const char*>(saved);
  const float* P = reinterpret_cast<const float*>(sv + o.s_p);
  const float* att = reinterpret_cast<const float*>(sv + o.s_att);
  float* Gm = reinterpret_cast<float*>(ws + o.w_g);
  float* dP = reinterpret_cast<float*>(ws + o.w_dp);
  float* dz = reinterpret_cast<float*>(ws + o.w_dz);
  float* dz_t = reinterpret_cast<float*>(ws + o.w_dzt);
  float* att_t = reinterpret_cast<float*>(ws + o.w_att_t);
  float* ds = reinterpret_cast<float*>(ws + o.w_dsdt);
  float* dt = ds + o.ld_n;
  const int32_t* erow = plan_erow(csr);
  GNN_HIP(mask_launch(n, h, h, Y, dY, layer->ld_y, Gm, o.ld_h, nullptr, 0, stream));
  if (nnz > 0) {
    timer_begin(GNN_K_SDDMM, stream);
    const unsigned grid = (unsigned)std::min<int64_t>(ceil_div(nnz, 16), 8192);
    if (h % 4 == 0)
      gat_sddmm_kernel<true><<<grid, 256, 0, stream>>>(nnz, h, erow, csr->indices, Gm,
                                                       o.ld_h, P, o.ld_h, att, alpha, dz);
    else
      gat_sddmm_kernel<false><<<grid, 256, 0, stream>>>(nnz, h, erow, csr->indices, Gm,
                                                        o.ld_h, P, o.ld_h, att, alpha, dz);
    timer_end(GNN_K_SDDMM, 8.0 * (double)nnz * h, stream);
    GNN_HIP(hipGetLastError());
    GNN_HIP(transpose_values_launch(n, nnz, csr->indptr, csr->indices, dz, dz_t,
                                    csr->plan, stream));
    GNN_HIP(transpose_values_launch(n, nnz, csr->indptr, csr->indices, att, att_t,
                                    csr->plan, stream));
  }
  gat_rowsums_kernel<<<(unsigned)ceil_div(n, 4), 256, 0, stream>>>(n, csr->indptr, dz,
                                                                    dz_t, ds, dt);
  GNN_HIP(hipGetLastError());
  // dP = A_att^T G, then the rank-2 terms of the scores
  SpmmCall c = spmm_call(csr, true, h, Gm, o.ld_h, dP, o.ld_h);
  c.vals = att_t;
  GNN_HIP(spmm_launch(c, stream));
  gat_rank2_kernel<<<(unsigned)ceil_div((int64_t)n * h, 256), 256, 0, stream>>>(
      n, h, ds, dt, a, dP, o.ld_h);
  GNN_HIP(hipGetLastError());
  // da1 = P^T ds, da2 = P^T dt (weighted column sums), dW = X^T dP,
  // dX = dP W^T
  float* cspart = reinterpret_cast<float*>(ws + o.w_cs);
  GNN_HIP(colsum2_launch(n, h, P, o.ld_h, ds, dt, da, da + h, cspart, stream));
  // the weight gradient's reduction, if any, runs in the input-gradient
  // launch, which takes the other workspace region
  GemmFixup held;
  GNN_HIP(gemm_launch(gemm1(1, 0, f_in, h, n, X, layer->ld_x, dP, o.ld_h, dW, h, 0,
                            layer->flags), ws + o.w_gemm, o.w_gemm_x - o.w_gemm, stream,
                      dX ? &held : nullptr));
  if (dX)
    GNN_HIP(gemm_launch(gemm1(0, 1, n, f_in, h, dP, o.ld_h, W, h, dX, layer->ld_dx, 0,
                              layer->flags), ws + o.w_gemm_x, o.total - o.w_gemm_x, stream,
                        nullptr, &held));
  return GNN_OK;
}

}  // extern "C"
