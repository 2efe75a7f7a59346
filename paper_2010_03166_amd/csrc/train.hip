// Classifier head, loss and weight update of a training iteration (Section
// 3.1, Eqs. "mlp forward" and "loss forward"; Algorithm 1; the gradients of
// Section 5.1):
//   XM = ReLU(X W)                          (matrix cores, ReLU in the epilogue)
//   Y  = softmax rows of XM  or  sigmoid(XM)
//   L  = mean over rows of the cross-entropy against the 0/1 targets T
//   G  = (Y - T) / n * 1[XM > 0]            (one wavefront per row)
//   dW = X^T G,  dX = G W^T                 (matrix cores)
// and the weight updates W -= lr g (SGD) or Adam.  The loss is summed in a
// fixed order (per block, then over blocks), so it is bit-reproducible.
#include <cmath>

#include "abi.hpp"

using namespace gnnprop;

namespace {

constexpr int LOSS_ROWS = 4;  // rows (wavefronts) per block

__device__ inline float wave_sum(float v) {
#pragma unroll
  for (int d = 32; d > 0; d >>= 1) v += __shfl_xor(v, d, 64);
  return v;
}
__device__ inline float wave_max(float v) {
#pragma unroll
  for (int d = 32; d > 0; d >>= 1) v = fmaxf(v, __shfl_xor(v, d, 64));
  return v;
}

// One wavefront per row; lanes stride over the C columns.  part[block]
// receives the block's rows' summed cross-entropy.
template <int KIND>
__global__ __launch_bounds__(64 * LOSS_ROWS) void loss_grad_kernel(
    int32_t n, int32_t C, const float* __restrict__ XM, int64_t ld_m,
    const float* __restrict__ T, int64_t ld_t, float* __restrict__ G,
    int64_t ld_g, float* __restrict__ probs, int64_t ld_p,
    float* __restrict__ part) {
  __shared__ float s_loss[LOSS_ROWS];
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int v = blockIdx.x * LOSS_ROWS + w;
  float row = 0.f;
  if (v < n) {
    const float* xm = XM + (int64_t)v * ld_m;
    const float* t = T + (int64_t)v * ld_t;
    float* g = G + (int64_t)v * ld_g;
    const float inv_n = 1.f / (float)n;
    if (KIND == GNN_LOSS_SOFTMAX) {
      float m = -INFINITY;
      for (int c = lane; c < C; c += 64) m = fmaxf(m, xm[c]);
      m = wave_max(m);
      float s = 0.f;
      for (int c = lane; c < C; c += 64) s += expf(xm[c] - m);
      const float ls = logf(wave_sum(s));
      for (int c = lane; c < C; c += 64) {
        const float x = xm[c];
        const float lp = x - m - ls;  // log Y
        const float y = expf(lp);
        row -= t[c] * lp;
        if (probs) probs[(int64_t)v * ld_p + c] = y;
        g[c] = x > 0.f ? (y - t[c]) * inv_n : 0.f;
      }
    } else {
      for (int c = lane; c < C; c += 64) {
        const float x = xm[c];
        const float e = expf(-x);
        const float y = 1.f / (1.f + e);
        const float l1 = -log1pf(e);  // log Y;  log(1 - Y) = l1 - x
        row -= t[c] * l1 + (1.f - t[c]) * (l1 - x);
        if (probs) probs[(int64_t)v * ld_p + c] = y;
        g[c] = x > 0.f ? (y - t[c]) * inv_n : 0.f;
      }
    }
    row = wave_sum(row);
  }
  if (lane == 0) s_loss[w] = row;
  __syncthreads();
  if (threadIdx.x == 0) {
    float s = 0.f;
    for (int k = 0; k < LOSS_ROWS; ++k) s += s_loss[k];
    part[blockIdx.x] = s;
  }
}

// Sums the block partials in block order (one block; each thread a strided
// subset, then a fixed tree), divides by n.
__global__ __launch_bounds__(256) void loss_final_kernel(
    int32_t nblk, int32_t n, const float* __restrict__ part,
    float* __restrict__ loss) {
  __shared__ float s[256];
  float acc = 0.f;
  for (int b = threadIdx.x; b < nblk; b += 256) acc += part[b];
  s[threadIdx.x] = acc;
  __syncthreads();
  for (int d = 128; d > 0; d >>= 1) {
    if ((int)threadIdx.x < d) s[threadIdx.x] += s[threadIdx.x + d];
    __syncthreads();
  }
  if (threadIdx.x == 0) *loss = n > 0 ? s[0] / (float)n : 0.f;
}

__global__ __launch_bounds__(256) void fill_zero_kernel(int64_t count,
                                                        float* __restrict__ p) {
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < count;
       i += (int64_t)gridDim.x * 256)
    p[i] = 0.f;
}

// The updates stream W, G (and m, v) once; with 16-byte aligned arrays a
// thread takes four consecutive weights per access (the tail singly).
template <bool VEC>
__global__ __launch_bounds__(256) void sgd_kernel(int64_t count, float* __restrict__ W,
                                                  const float* __restrict__ g, float lr) {
  const int64_t stride = (int64_t)gridDim.x * 256;
  int64_t i0 = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (VEC) {
    const int64_t c4 = count >> 2;
    for (int64_t i = i0; i < c4; i += stride) {
      float4 w = reinterpret_cast<float4*>(W)[i];
      const float4 d = reinterpret_cast<const float4*>(g)[i];
      w.x -= lr * d.x;
      w.y -= lr * d.y;
      w.z -= lr * d.z;
      w.w -= lr * d.w;
      reinterpret_cast<float4*>(W)[i] = w;
    }
    i0 += c4 << 2;
  }
  for (int64_t i = i0; i < count; i += stride) W[i] -= lr * g[i];
}

struct AdamCoef {
  float lr, b1, omb1, b2, omb2, eps, c1, c2;
};

__device__ inline void adam_one(float& w, float gi, float& m, float& v, const AdamCoef& a) {
  m = a.b1 * m + a.omb1 * gi;
  v = a.b2 * v + a.omb2 * gi * gi;
  w -= a.lr * (m / a.c1) / (sqrtf(v / a.c2) + a.eps);
}

template <bool VEC>
__global__ __launch_bounds__(256) void adam_kernel(int64_t count, float* __restrict__ W,
                                                   const float* __restrict__ g,
                                                   float* __restrict__ m,
                                                   float* __restrict__ v, AdamCoef a) {
  const int64_t stride = (int64_t)gridDim.x * 256;
  int64_t i0 = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (VEC) {
    const int64_t c4 = count >> 2;
    for (int64_t i = i0; i < c4; i += stride) {
      float4 w = reinterpret_cast<float4*>(W)[i];
      const float4 d = reinterpret_cast<const float4*>(g)[i];
      float4 mm = reinterpret_cast<float4*>(m)[i];
      float4 vv = reinterpret_cast<float4*>(v)[i];
      adam_one(w.x, d.x, mm.x, vv.x, a);
      adam_one(w.y, d.y, mm.y, vv.y, a);
      adam_one(w.z, d.z, mm.z, vv.z, a);
      adam_one(w.w, d.w, mm.w, vv.w, a);
      reinterpret_cast<float4*>(W)[i] = w;
      reinterpret_cast<float4*>(m)[i] = mm;
      reinterpret_cast<float4*>(v)[i] = vv;
    }
    i0 += c4 << 2;
  }
  for (int64_t i = i0; i < count; i += stride) {
    float w = W[i], mi = m[i], vi = v[i];
    adam_one(w, g[i], mi, vi, a);
    W[i] = w;
    m[i] = mi;
    v[i] = vi;
  }
}

inline bool al16(const void* p) { return reinterpret_cast<uintptr_t>(p) % 16 == 0; }

inline unsigned update_grid(int64_t count) {
  return (unsigned)std::max<int64_t>(1, std::min<int64_t>(ceil_div(count, 1024), 2048));
}

struct ClsLayout {
  int64_t ld_c;
  int nblk;
  // GEMM workspace: [off_gemm, off_gemm_x) the weight gradient's partial
  // tiles, summed by the input-gradient launch; [off_gemm_x, total) the rest
  size_t off_m, off_g, off_part, off_gemm, off_gemm_x, total;
};

GemmBatch prod(int ta, int tb, int32_t M, int32_t N, int32_t K, const float* A,
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

ClsLayout cls_layout(int32_t n, int32_t f, int32_t C, uint32_t flags) {
  ClsLayout o;
  o.ld_c = round_up(C, 4);
  o.nblk = (int)std::max<int64_t>(1, ceil_div(n, LOSS_ROWS));
  const size_t gw = gemm_workspace_bytes(prod(1, 0, f, C, n, 0, f, 0, C, 0, C, 0, flags));
  const size_t g =
      std::max(gemm_workspace_bytes(prod(0, 0, n, C, f, 0, f, 0, C, 0, C, 1, flags)),
               gemm_workspace_bytes(prod(0, 1, n, f, C, 0, C, 0, C, 0, f, 0, flags)));
  o.off_m = 0;
  o.off_g = round_up((size_t)n * o.ld_c * 4, 256);
  o.off_part = o.off_g + round_up((size_t)n * o.ld_c * 4, 256);
  o.off_gemm = o.off_part + round_up((size_t)o.nblk * 4, 256);
  o.off_gemm_x = o.off_gemm + round_up(gw, 256);
  o.total = o.off_gemm_x + round_up(g, 256);
  return o;
}

}  // namespace

extern "C" {

size_t gnn_classifier_workspace_bytes(int32_t n, int32_t f, int32_t C) {
  if (n < 0 || f <= 0 || C <= 0) return 0;
  // the largest need of the three product modes (their work splits differ)
  size_t need = 0;
  for (const uint32_t flags : {0u, GNN_FLAG_BF16, GNN_FLAG_F32_MFMA})
    need = std::max(need, cls_layout(n, f, C, flags).total);
  return need;
}

gnn_status gnn_classifier(int32_t n, int32_t f, int32_t C, int32_t kind,
                          uint32_t flags, const float* X, int64_t ld_x,
                          const float* W, const float* T, int64_t ld_t,
                          float* xm, int64_t ld_xm, float* probs, int64_t ld_p,
                          float* loss, float* dW, float* dX, int64_t ld_dx,
                          void* workspace, size_t workspace_bytes,
                          hipStream_t stream) {
  if (n < 0 || f <= 0 || C <= 0) return GNN_ERR_SHAPE;
  if (kind != GNN_LOSS_SOFTMAX && kind != GNN_LOSS_SIGMOID) return GNN_ERR_UNSUPPORTED;
  if ((flags & ~GEMM_FLAGS) || !gemm_flags_ok(flags)) return GNN_ERR_UNSUPPORTED;
  if (!W || !loss || !dW) return GNN_ERR_NULL;
  if (n > 0 && (!X || !T)) return GNN_ERR_NULL;
  if (ld_x < f || ld_t < C || (xm && ld_xm < C) || (probs && ld_p < C) ||
      (dX && ld_dx < f))
    return GNN_ERR_SHAPE;
  if (!buf16(workspace)) return GNN_ERR_UNSUPPORTED;
  const ClsLayout o = cls_layout(n, f, C, flags);
  if (workspace_bytes < o.total || !workspace) return GNN_ERR_WORKSPACE;
  {
    const void* ins[] = {X, W, T};
    const size_t inb[] = {mat_bytes(n, f, ld_x), (size_t)f * C * 4, mat_bytes(n, C, ld_t)};
    const void* outs[] = {xm, probs, loss, dW, dX, workspace};
    const size_t outb[] = {xm ? mat_bytes(n, C, ld_xm) : 0,
                           probs ? mat_bytes(n, C, ld_p) : 0, 4, (size_t)f * C * 4,
                           dX ? mat_bytes(n, f, ld_dx) : 0, o.total};
    for (int i = 0; i < 6; ++i) {
      for (int k = 0; k < 3; ++k)
        if (ranges_overlap(outs[i], outb[i], ins[k], inb[k])) return GNN_ERR_ALIAS;
      for (int k = 0; k < i; ++k)
        if (ranges_overlap(outs[i], outb[i], outs[k], outb[k])) return GNN_ERR_ALIAS;
    }
  }
  char* ws = static_cast<char*>(workspace);
  float* XM = xm ? xm : reinterpret_cast<float*>(ws + o.off_m);
  const int64_t ld_m = xm ? ld_xm : o.ld_c;
  float* G = reinterpret_cast<float*>(ws + o.off_g);
  float* part = reinterpret_cast<float*>(ws + o.off_part);
  void* gws = ws + o.off_gemm;
  const size_t gws_bytes = o.total - o.off_gemm;
  if (n > 0) {
    GNN_HIP(gemm_launch(prod(0, 0, n, C, f, X, ld_x, W, C, XM, ld_m, 1, flags), gws,
                        gws_bytes, stream));
    timer_begin(GNN_K_LOSS, stream);
    if (kind == GNN_LOSS_SOFTMAX)
      loss_grad_kernel<GNN_LOSS_SOFTMAX><<<o.nblk, 64 * LOSS_ROWS, 0, stream>>>(
          n, C, XM, ld_m, T, ld_t, G, o.ld_c, probs, ld_p, part);
    else
      loss_grad_kernel<GNN_LOSS_SIGMOID><<<o.nblk, 64 * LOSS_ROWS, 0, stream>>>(
          n, C, XM, ld_m, T, ld_t, G, o.ld_c, probs, ld_p, part);
  }
  loss_final_kernel<<<1, 256, 0, stream>>>(n > 0 ? o.nblk : 0, n, part, loss);
  if (n > 0) timer_end(GNN_K_LOSS, 12.0 * n * C, stream);
  GNN_HIP(hipGetLastError());
  if (n == 0) {  // no rows: zero gradient (a kernel, so graph capture works)
    const int64_t cnt = (int64_t)f * C;
    fill_zero_kernel<<<(unsigned)std::min<int64_t>(ceil_div(cnt, 256), 4096), 256, 0,
                       stream>>>(cnt, dW);
    GNN_HIP(hipGetLastError());
    return GNN_OK;
  }
  // the weight gradient's reduction, if any, runs in the input-gradient
  // launch, which takes the other workspace region
  GemmFixup held;
  GNN_HIP(gemm_launch(prod(1, 0, f, C, n, X, ld_x, G, o.ld_c, dW, C, 0, flags), gws,
                      o.off_gemm_x - o.off_gemm, stream, dX ? &held : nullptr));
  if (dX)
    GNN_HIP(gemm_launch(prod(0, 1, n, f, C, G, o.ld_c, W, C, dX, ld_dx, 0, flags),
                        ws + o.off_gemm_x, o.total - o.off_gemm_x, stream, nullptr, &held));
  return GNN_OK;
}

gnn_status gnn_sgd_step(int64_t count, float* W, const float* G, double lr,
                        hipStream_t stream) {
  if (count < 0) return GNN_ERR_SHAPE;
  if (count == 0) return GNN_OK;
  if (!W || !G) return GNN_ERR_NULL;
  if (ranges_overlap(W, (size_t)count * 4, G, (size_t)count * 4)) return GNN_ERR_ALIAS;
  const unsigned grid = update_grid(count);
  timer_begin(GNN_K_UPDATE, stream);
  if (al16(W) && al16(G))
    sgd_kernel<true><<<grid, 256, 0, stream>>>(count, W, G, (float)lr);
  else
    sgd_kernel<false><<<grid, 256, 0, stream>>>(count, W, G, (float)lr);
  timer_end(GNN_K_UPDATE, 12.0 * count, stream);
  GNN_HIP(hipGetLastError());
  return GNN_OK;
}

gnn_status gnn_adam_step(int64_t count, float* W, const float* G, float* m,
                         float* v, double lr, double beta1, double beta2,
                         double eps, int32_t t, hipStream_t stream) {
  if (count < 0 || t < 1) return GNN_ERR_SHAPE;
  if (count == 0) return GNN_OK;
  if (!W || !G || !m || !v) return GNN_ERR_NULL;
  const size_t b = (size_t)count * 4;
  if (ranges_overlap(W, b, G, b) || ranges_overlap(m, b, v, b) ||
      ranges_overlap(W, b, m, b) || ranges_overlap(W, b, v, b) ||
      ranges_overlap(G, b, m, b) || ranges_overlap(G, b, v, b))
    return GNN_ERR_ALIAS;
  // the coefficients in double, each rounded once to fp32
  const float c1 = (float)(1.0 - std::pow(beta1, t));
  const float c2 = (float)(1.0 - std::pow(beta2, t));
  const AdamCoef a{(float)lr, (float)beta1, (float)(1.0 - beta1), (float)beta2,
                   (float)(1.0 - beta2), (float)eps, c1, c2};
  const unsigned grid = update_grid(count);
  timer_begin(GNN_K_UPDATE, stream);
  if (al16(W) && al16(G) && al16(m) && al16(v))
    adam_kernel<true><<<grid, 256, 0, stream>>>(count, W, G, m, v, a);
  else
    adam_kernel<false><<<grid, 256, 0, stream>>>(count, W, G, m, v, a);
  timer_end(GNN_K_UPDATE, 28.0 * count, stream);
  GNN_HIP(hipGetLastError());
  return GNN_OK;
}

}  // extern "C"
