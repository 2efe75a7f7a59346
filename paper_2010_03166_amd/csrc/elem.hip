// Elementwise pieces of the backward pass: the ReLU mask applied to the
// output gradient (mask() in Section 5.1, Eq. "gcn backward") and the
// column sums that give the bias gradients.
#include "internal.hpp"

namespace gnnprop {

// G = dY * 1[Y > 0] over n x width; columns [0, split) go to dst0, the rest
// to dst1 (the self and neighbour halves of a GraphSAGE output, or one block
// when split = width).  One thread per 4 columns when every row start is
// aligned for them.  H0: dst0 holds bf16 (rounded to nearest even).
template <bool VEC, bool H0>
__global__ __launch_bounds__(256) void mask_kernel(
    int32_t n, int32_t width, int32_t split, const float* __restrict__ Y,
    const float* __restrict__ dY, int64_t ld_y, void* __restrict__ dst0,
    int64_t ld0, float* __restrict__ dst1, int64_t ld1) {
  constexpr int W = VEC ? 4 : 1;
  const int per_row = width / W;
  const int64_t total = (int64_t)n * per_row;
  for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < total;
       e += (int64_t)gridDim.x * blockDim.x) {
    const int row = (int)(e / per_row);
    const int col = (int)(e % per_row) * W;
    const int64_t src = (int64_t)row * ld_y + col;
    const bool first = col < split;
    const int64_t at = first ? (int64_t)row * ld0 + col : (int64_t)row * ld1 + (col - split);
    if (VEC) {
      const float4 y = *reinterpret_cast<const float4*>(Y + src);
      const float4 d = *reinterpret_cast<const float4*>(dY + src);
      float4 g;
      g.x = y.x > 0.f ? d.x : 0.f;
      g.y = y.y > 0.f ? d.y : 0.f;
      g.z = y.z > 0.f ? d.z : 0.f;
      g.w = y.w > 0.f ? d.w : 0.f;
      if (H0 && first)
        *reinterpret_cast<uint2*>(static_cast<uint16_t*>(dst0) + at) =
            make_uint2(pack_bf16(g.x, g.y), pack_bf16(g.z, g.w));
      else
        *reinterpret_cast<float4*>((first ? static_cast<float*>(dst0) : dst1) + at) = g;
    } else {
      const float g = Y[src] > 0.f ? dY[src] : 0.f;
      if (H0 && first)
        static_cast<uint16_t*>(dst0)[at] = (uint16_t)(pack_bf16(g, 0.f) & 0xffffu);
      else
        (first ? static_cast<float*>(dst0) : dst1)[at] = g;
    }
  }
}

hipError_t mask_launch(int32_t n, int32_t width, int32_t split,
                       const float* Y, const float* dY, int64_t ld_y,
                       void* dst0, int64_t ld0, float* dst1, int64_t ld1,
                       hipStream_t s, bool dst0_bf16) {
  if (n <= 0 || width <= 0) return hipSuccess;
  const bool d0_ok = dst0_bf16 ? (reinterpret_cast<uintptr_t>(dst0) % 8 == 0 && ld0 % 4 == 0)
                               : vec4_ok(dst0, ld0);
  const bool vec = (width % 4 == 0) && (split % 4 == 0) && vec4_ok(Y, ld_y) &&
                   vec4_ok(dY, ld_y) && d0_ok && (split == width || vec4_ok(dst1, ld1));
  const int64_t units = (int64_t)n * width / (vec ? 4 : 1);
  const unsigned grid = (unsigned)std::min<int64_t>(ceil_div(units, 256), 8192);
  timer_begin(GNN_K_MASK, s);
  if (vec && dst0_bf16)
    mask_kernel<true, true><<<grid, 256, 0, s>>>(n, width, split, Y, dY, ld_y, dst0, ld0, dst1, ld1);
  else if (vec)
    mask_kernel<true, false><<<grid, 256, 0, s>>>(n, width, split, Y, dY, ld_y, dst0, ld0, dst1, ld1);
  else if (dst0_bf16)
    mask_kernel<false, true><<<grid, 256, 0, s>>>(n, width, split, Y, dY, ld_y, dst0, ld0, dst1, ld1);
  else
    mask_kernel<false, false><<<grid, 256, 0, s>>>(n, width, split, Y, dY, ld_y, dst0, ld0, dst1, ld1);
  // Y and dY read (8 bytes per element), G written: columns [0, split) as
  // bf16 when dst0_bf16, the rest as fp32
  timer_end(GNN_K_MASK,
            8.0 * n * width + (dst0_bf16 ? 2.0 : 4.0) * n * split + 4.0 * n * (width - split),
            s);
  return hipGetLastError();
}

// Column sums in two deterministic phases.  Phase 1: block (rb, cb) covers
// 64 columns and CS_ROWS rows; each of its 4 waves takes CS_RPT consecutive
// rows, issuing all of their loads before the adds (the sum is latency
// bound otherwise), and the wave sums are combined in wave order.  Phase 2:
// per CS_FC columns, CS_FG thread groups each add a contiguous share of the
// row-block partials in ascending order (a few loads in flight per thread,
// so the pass is one memory round trip or two), combined in group order.
// NW = 2 forms two weighted sums (weights w0[r], w1[r]) from one pass over G.
constexpr int CS_RPT = 16;
constexpr int CS_ROWS = 4 * CS_RPT;
constexpr int CS_FC = 16, CS_FG = 256 / CS_FC;

// MASKED: the summed value is G[r, c] where Ym[r, c] > 0, else 0 (Ym has
// G's row stride).
template <int NW, bool MASKED>
__global__ __launch_bounds__(256) void colsum_partial_kernel(
    int32_t n, int32_t w, const float* __restrict__ G, int64_t ldg,
    const float* __restrict__ w0, const float* __restrict__ w1,
    float* __restrict__ part, int64_t pstride, const float* __restrict__ Ym) {
  __shared__ float s[NW][4][64];
  const int l = threadIdx.x & 63;
  const int grp = threadIdx.x >> 6;
  const int c = blockIdx.y * 64 + l;
  const int r0 = blockIdx.x * CS_ROWS + grp * CS_RPT;
  float acc[NW];
#pragma unroll
  for (int j = 0; j < NW; ++j) acc[j] = 0.f;
  if (c < w) {
    float v[CS_RPT];
#pragma unroll
    for (int k = 0; k < CS_RPT; ++k) {
      v[k] = r0 + k < n ? G[(int64_t)(r0 + k) * ldg + c] : 0.f;
      if (MASKED && r0 + k < n && !(Ym[(int64_t)(r0 + k) * ldg + c] > 0.f)) v[k] = 0.f;
    }
#pragma unroll
    for (int k = 0; k < CS_RPT; ++k) {
      if (r0 + k >= n) break;
      acc[0] += w0 ? w0[r0 + k] * v[k] : v[k];
      if (NW == 2) acc[NW - 1] += w1[r0 + k] * v[k];
    }
  }
#pragma unroll
  for (int j = 0; j < NW; ++j) s[j][grp][l] = acc[j];
  __syncthreads();
  if (grp == 0 && c < w) {
#pragma unroll
    for (int j = 0; j < NW; ++j)
      part[j * pstride + (int64_t)blockIdx.x * w + c] =
          ((s[j][0][l] + s[j][1][l]) + s[j][2][l]) + s[j][3][l];
  }
}

template <int NW>
__global__ __launch_bounds__(256) void colsum_final_kernel(
    int32_t nblk, int32_t w, const float* __restrict__ part, int64_t pstride,
    float* __restrict__ out0, float* __restrict__ out1) {
  __shared__ float s[NW][CS_FG][CS_FC];
  const int l = threadIdx.x % CS_FC;
  const int grp = threadIdx.x / CS_FC;
  const int c = blockIdx.x * CS_FC + l;
  const int q = (nblk + CS_FG - 1) / CS_FG;
  const int b0 = min(nblk, grp * q), b1 = min(nblk, b0 + q);
#pragma unroll
  for (int j = 0; j < NW; ++j) {
    float acc = 0.f;
    if (c < w) {
      const float* p = part + j * pstride + c;
#pragma unroll 8
      for (int b = b0; b < b1; ++b) acc += p[(int64_t)b * w];
    }
    s[j][grp][l] = acc;
  }
  __syncthreads();
  if (threadIdx.x < CS_FC && c < w) {
#pragma unroll
    for (int j = 0; j < NW; ++j) {
      float acc = s[j][0][l];
      for (int g = 1; g < CS_FG; ++g) acc += s[j][g][l];
      (j == 0 ? out0 : out1)[c] = acc;
    }
  }
}

size_t colsum_partials_bytes(int32_t n, int32_t w, int nw) {
  return round_up((size_t)nw * std::max<int64_t>(1, ceil_div(n, CS_ROWS)) * w * 4, 256);
}

hipError_t colsum_launch(int32_t n, int32_t w, const float* G, int64_t ldg,
                         float* out, float* partials, hipStream_t s,
                         const float* row_weight) {
  if (w <= 0) return hipSuccess;
  const int nblk = (int)std::max<int64_t>(1, ceil_div(n, CS_ROWS));
  const int64_t ps = (int64_t)nblk * w;
  dim3 grid((unsigned)nblk, (unsigned)ceil_div(w, 64));
  timer_begin(GNN_K_COLSUM, s);
  colsum_partial_kernel<1, false><<<grid, 256, 0, s>>>(n, w, G, ldg, row_weight, nullptr,
                                                       partials, ps, nullptr);
  colsum_final_kernel<1><<<(unsigned)ceil_div(w, CS_FC), 256, 0, s>>>(nblk, w, partials, ps,
                                                                       out, nullptr);
  timer_end(GNN_K_COLSUM, 4.0 * n * w, s);
  return hipGetLastError();
}

hipError_t colsum2_launch(int32_t n, int32_t w, const float* G, int64_t ldg,
                          const float* w0, const float* w1, float* out0,
                          float* out1, float* partials, hipStream_t s) {
  if (w <= 0) return hipSuccess;
  const int nblk = (int)std::max<int64_t>(1, ceil_div(n, CS_ROWS));
  const int64_t ps = (int64_t)nblk * w;
  dim3 grid((unsigned)nblk, (unsigned)ceil_div(w, 64));
  timer_begin(GNN_K_COLSUM, s);
  colsum_partial_kernel<2, false><<<grid, 256, 0, s>>>(n, w, G, ldg, w0, w1, partials, ps,
                                                       nullptr);
  colsum_final_kernel<2><<<(unsigned)ceil_div(w, CS_FC), 256, 0, s>>>(nblk, w, partials, ps,
                                                                       out0, out1);
  timer_end(GNN_K_COLSUM, 4.0 * n * w + 8.0 * n, s);
  return hipGetLastError();
}

hipError_t colsum_masked_launch(int32_t n, int32_t w, const float* Y, const float* dY,
                                int64_t ld, float* out, float* partials, hipStream_t s) {
  if (w <= 0) return hipSuccess;
  const int nblk = (int)std::max<int64_t>(1, ceil_div(n, CS_ROWS));
  const int64_t ps = (int64_t)nblk * w;
  dim3 grid((unsigned)nblk, (unsigned)ceil_div(w, 64));
  timer_begin(GNN_K_COLSUM, s);
  colsum_partial_kernel<1, true><<<grid, 256, 0, s>>>(n, w, dY, ld, nullptr, nullptr, partials,
                                                      ps, Y);
  colsum_final_kernel<1><<<(unsigned)ceil_div(w, CS_FC), 256, 0, s>>>(nblk, w, partials, ps,
                                                                       out, nullptr);
  timer_end(GNN_K_COLSUM, 8.0 * n * w, s);
  return hipGetLastError();
}

}  // namespace gnnprop
