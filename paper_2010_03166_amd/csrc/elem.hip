// Elementwise pieces of the backward pass: the ReLU mask applied to the
// output gradient (mask() in Section 5.1, Eq. "gcn backward") and the
// column sums that give the bias gradients.
#include "internal.hpp"

namespace gnnprop {

// G = dY * 1[Y > 0] over n x width; columns [0, split) go to dst0, the rest
// to dst1 (the self and neighbour halves of a GraphSAGE output, or one block
// when split = width).  One thread per 4 columns when every row start is
// 16-byte aligned.
template <bool VEC>
__global__ __launch_bounds__(256) void mask_kernel(
    int32_t n, int32_t width, int32_t split, const float* __restrict__ Y,
    const float* __restrict__ dY, int64_t ld_y, float* __restrict__ dst0,
    int64_t ld0, float* __restrict__ dst1, int64_t ld1) {
  constexpr int W = VEC ? 4 : 1;
  const int per_row = width / W;
  const int64_t total = (int64_t)n * per_row;
  for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < total;
       e += (int64_t)gridDim.x * blockDim.x) {
    const int row = (int)(e / per_row);
    const int col = (int)(e % per_row) * W;
    const int64_t src = (int64_t)row * ld_y + col;
    float* dst = col < split ? dst0 + (int64_t)row * ld0 + col
                             : dst1 + (int64_t)row * ld1 + (col - split);
    if (VEC) {
      const float4 y = *reinterpret_cast<const float4*>(Y + src);
      const float4 d = *reinterpret_cast<const float4*>(dY + src);
      float4 g;
      g.x = y.x > 0.f ? d.x : 0.f;
      g.y = y.y > 0.f ? d.y : 0.f;
      g.z = y.z > 0.f ? d.z : 0.f;
      g.w = y.w > 0.f ? d.w : 0.f;
      *reinterpret_cast<float4*>(dst) = g;
    } else {
      *dst = Y[src] > 0.f ? dY[src] : 0.f;
    }
  }
}

hipError_t mask_launch(int32_t n, int32_t width, int32_t split,
                       const float* Y, const float* dY, int64_t ld_y,
                       float* dst0, int64_t ld0, float* dst1, int64_t ld1,
                       hipStream_t s) {
  if (n <= 0 || width <= 0) return hipSuccess;
  const bool vec = (width % 4 == 0) && (split % 4 == 0) && vec4_ok(Y, ld_y) &&
                   vec4_ok(dY, ld_y) && vec4_ok(dst0, ld0) &&
                   (split == width || vec4_ok(dst1, ld1));
  const int64_t units = (int64_t)n * width / (vec ? 4 : 1);
  const unsigned grid = (unsigned)std::min<int64_t>(ceil_div(units, 256), 8192);
  timer_begin(GNN_K_MASK, s);
  if (vec)
    mask_kernel<true><<<grid, 256, 0, s>>>(n, width, split, Y, dY, ld_y, dst0, ld0, dst1, ld1);
  else
    mask_kernel<false><<<grid, 256, 0, s>>>(n, width, split, Y, dY, ld_y, dst0, ld0, dst1, ld1);
  timer_end(GNN_K_MASK, 12.0 * n * width, s);
  return hipGetLastError();
}

// Column sums in two deterministic phases: block (cb, rb) sums rows
// [256 rb, 256 rb + 256) of 64 columns (4 row groups of 64 rows, combined in
// group order), then one thread per column adds the row-block partials in
// ascending rb.
constexpr int CS_ROWS = 256;

__global__ __launch_bounds__(256) void colsum_partial_kernel(
    int32_t n, int32_t w, const float* __restrict__ G, int64_t ldg,
    float* __restrict__ part) {
  __shared__ float s[4][64];
  const int c = blockIdx.x * 64 + (threadIdx.x & 63);
  const int grp = threadIdx.x >> 6;
  const int r0 = blockIdx.y * CS_ROWS + grp * (CS_ROWS / 4);
  float acc = 0.f;
  if (c < w)
    for (int r = r0; r < min(n, r0 + CS_ROWS / 4); ++r)
      acc += G[(int64_t)r * ldg + c];
  s[grp][threadIdx.x & 63] = acc;
  __syncthreads();
  if (grp == 0 && c < w) {
    const int l = threadIdx.x & 63;
    part[(int64_t)blockIdx.y * w + c] = ((s[0][l] + s[1][l]) + s[2][l]) + s[3][l];
  }
}

__global__ __launch_bounds__(256) void colsum_final_kernel(
    int32_t nblk, int32_t w, const float* __restrict__ part,
    float* __restrict__ out) {
  const int c = blockIdx.x * blockDim.x + threadIdx.x;
  if (c >= w) return;
  float acc = 0.f;
  for (int b = 0; b < nblk; ++b) acc += part[(int64_t)b * w + c];
  out[c] = acc;
}

size_t colsum_partials_bytes(int32_t n, int32_t w) {
  return round_up((size_t)std::max<int64_t>(1, ceil_div(n, CS_ROWS)) * w * 4, 256);
}

hipError_t colsum_launch(int32_t n, int32_t w, const float* G, int64_t ldg,
                         float* out, float* partials, hipStream_t s) {
  if (w <= 0) return hipSuccess;
  const int nblk = (int)std::max<int64_t>(1, ceil_div(n, CS_ROWS));
  dim3 grid((unsigned)ceil_div(w, 64), (unsigned)nblk);
  timer_begin(GNN_K_COLSUM, s);
  colsum_partial_kernel<<<grid, 256, 0, s>>>(n, w, G, ldg, partials);
  colsum_final_kernel<<<(unsigned)ceil_div(w, 256), 256, 0, s>>>(nblk, w, partials, out);
  timer_end(GNN_K_COLSUM, 4.0 * n * w, s);
  return hipGetLastError();
}

}  // namespace gnnprop
