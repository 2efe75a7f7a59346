// Dense weight transformation on the gfx950 matrix cores (the second of the
// three kernels of Section 5.1).
//
// C = sum_s op(A_s) op(B_s) (+ bias, ReLU), fp32 in and out, on
// v_mfma_f32_32x32x2_f32.  A block of 256 threads (4 wavefronts in 2 x 2)
// owns a 128 x 128 output tile; each wavefront holds a 64 x 64 sub-tile as
// 2 x 2 MFMA accumulators (64 accumulator registers per lane).  K advances
// in 32-deep slices staged through double-buffered LDS: while the matrix
// cores consume slice k, the global loads of slice k+1 are in flight, and
// one barrier per slice separates the two buffers.  Both operands live in
// LDS as [k][m] / [k][n] rows, so every MFMA operand read is 32 consecutive
// floats per half-wavefront; operands stored the other way round are
// transposed on their way into LDS.  Shapes with few output tiles (the
// weight gradients, K = n) are split along K; the partial tiles are summed
// in split order by a second kernel, so results are deterministic.
#include "internal.hpp"

namespace gnnprop {

typedef float floatx16 __attribute__((ext_vector_type(16)));

constexpr int BM = 128, BN = 128, BK = 32;
constexpr int LDS_STRIDE = 160;  // floats per LDS row: 128 + 32 padding

struct GemmKArgs {
  GemmProblem p[2];
  int32_t nprob;
  int32_t tiles_m[2];
  int32_t tile_start[2];
  int32_t ktiles0[2];  // K slices of segment 0
  int32_t ktiles[2];   // K slices over all segments
  int32_t total_tiles;
  int32_t splits;
  float* part[2];
  int32_t vec_a, vec_b;
};

// Element (r, c..c+3) of a row-major R x C matrix with row stride ld; zeros
// outside the matrix.
__device__ inline float4 load4(const float* base, int64_t ld, int r, int c,
                               int R, int C, bool vec) {
  float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
  if (r < R && c < C) {
    const float* p = base + (int64_t)r * ld + c;
    if (vec && c + 3 < C) {
      v = *reinterpret_cast<const float4*>(p);
    } else {
      v.x = p[0];
      if (c + 1 < C) v.y = p[1];
      if (c + 2 < C) v.z = p[2];
      if (c + 3 < C) v.w = p[3];
    }
  }
  return v;
}

template <bool AT, bool BT>
__global__ __launch_bounds__(256, 2) void gemm_f32_kernel(GemmKArgs g) {
  __shared__ float As[2][BK][LDS_STRIDE];
  __shared__ float Bs[2][BK][LDS_STRIDE];

  const int tid = threadIdx.x;
  const int split = blockIdx.x / g.total_tiles;
  int t = blockIdx.x % g.total_tiles;
  const int pi = (g.nprob > 1 && t >= g.tile_start[1]) ? 1 : 0;
  t -= pi ? g.tile_start[1] : 0;

  // Problem fields, selected without dynamic indexing.
  const GemmProblem& P0 = g.p[0];
  const GemmProblem& P1 = g.p[1];
  const int M = pi ? P1.M : P0.M;
  const int N = pi ? P1.N : P0.N;
  const int tiles_m = pi ? g.tiles_m[1] : g.tiles_m[0];
  const int kt0 = pi ? g.ktiles0[1] : g.ktiles0[0];
  const int ktiles = pi ? g.ktiles[1] : g.ktiles[0];
  const float* A0 = pi ? P1.seg[0].A : P0.seg[0].A;
  const float* A1 = pi ? P1.seg[1].A : P0.seg[1].A;
  const float* B0 = pi ? P1.seg[0].B : P0.seg[0].B;
  const float* B1 = pi ? P1.seg[1].B : P0.seg[1].B;
  const int64_t lda0 = pi ? P1.seg[0].lda : P0.seg[0].lda;
  const int64_t lda1 = pi ? P1.seg[1].lda : P0.seg[1].lda;
  const int64_t ldb0 = pi ? P1.seg[0].ldb : P0.seg[0].ldb;
  const int64_t ldb1 = pi ? P1.seg[1].ldb : P0.seg[1].ldb;
  const int K0 = pi ? P1.seg[0].K : P0.seg[0].K;
  const int K1 = pi ? P1.seg[1].K : P0.seg[1].K;

  const int m0 = (t % tiles_m) * BM;
  const int n0 = (t / tiles_m) * BN;
  const int kt_per = (ktiles + g.splits - 1) / g.splits;
  const int kt_begin = min(ktiles, split * kt_per);
  const int kt_end = min(ktiles, kt_begin + kt_per);
  const bool va = g.vec_a != 0, vb = g.vec_b != 0;

  float4 ra[4], rb[4];
  auto load_slice = [&](int gt) {
    const bool s1 = gt >= kt0;
    const int k0 = (s1 ? gt - kt0 : gt) * BK;
    const float* A = s1 ? A1 : A0;
    const float* B = s1 ? B1 : B0;
    const int64_t lda = s1 ? lda1 : lda0;
    const int64_t ldb = s1 ? ldb1 : ldb0;
    const int K = s1 ? K1 : K0;
#pragma unroll
    for (int p = 0; p < 4; ++p) {
      if (!AT) {  // A is M x K row-major: 8 float4 per tile row
        const int row = (tid >> 3) + 32 * p, kq = tid & 7;
        ra[p] = load4(A, lda, m0 + row, k0 + 4 * kq, M, K, va);
      } else {    // A stored K x M
        const int kk = (tid >> 5) + 8 * p, mq = tid & 31;
        ra[p] = load4(A, lda, k0 + kk, m0 + 4 * mq, K, M, va);
      }
      if (!BT) {  // B is K x N row-major
        const int kk = (tid >> 5) + 8 * p, nq = tid & 31;
        rb[p] = load4(B, ldb, k0 + kk, n0 + 4 * nq, K, N, vb);
      } else {    // B stored N x K
        const int col = (tid >> 3) + 32 * p, kq = tid & 7;
        rb[p] = load4(B, ldb, n0 + col, k0 + 4 * kq, N, K, vb);
      }
    }
  };
  auto store_slice = [&](int buf) {
#pragma unroll
    for (int p = 0; p < 4; ++p) {
      if (!AT) {
        const int row = (tid >> 3) + 32 * p, kq = tid & 7;
        As[buf][4 * kq + 0][row] = ra[p].x;
        As[buf][4 * kq + 1][row] = ra[p].y;
        As[buf][4 * kq + 2][row] = ra[p].z;
        As[buf][4 * kq + 3][row] = ra[p].w;
      } else {
        const int kk = (tid >> 5) + 8 * p, mq = tid & 31;
        *reinterpret_cast<float4*>(&As[buf][kk][4 * mq]) = ra[p];
      }
      if (!BT) {
        const int kk = (tid >> 5) + 8 * p, nq = tid & 31;
        *reinterpret_cast<float4*>(&Bs[buf][kk][4 * nq]) = rb[p];
      } else {
        const int col = (tid >> 3) + 32 * p, kq = tid & 7;
        Bs[buf][4 * kq + 0][col] = rb[p].x;
        Bs[buf][4 * kq + 1][col] = rb[p].y;
        Bs[buf][4 * kq + 2][col] = rb[p].z;
        Bs[buf][4 * kq + 3][col] = rb[p].w;
      }
    }
  };

  const int wave = tid >> 6, lane = tid & 63;
  const int wm = wave & 1, wn = wave >> 1;
  const int lr = lane & 31, lk = lane >> 5;

  floatx16 acc[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

  if (kt_begin < kt_end) load_slice(kt_begin);
  int buf = 0;
  for (int gt = kt_begin; gt < kt_end; ++gt) {
    store_slice(buf);
    __syncthreads();
    if (gt + 1 < kt_end) load_slice(gt + 1);
#pragma unroll
    for (int s = 0; s < BK / 2; ++s) {
      const int kr = 2 * s + lk;
      const float a0 = As[buf][kr][wm * 64 + lr];
      const float a1 = As[buf][kr][wm * 64 + 32 + lr];
      const float b0 = Bs[buf][kr][wn * 64 + lr];
      const float b1 = Bs[buf][kr][wn * 64 + 32 + lr];
      acc[0][0] = __builtin_amdgcn_mfma_f32_32x32x2f32(a0, b0, acc[0][0], 0, 0, 0);
      acc[0][1] = __builtin_amdgcn_mfma_f32_32x32x2f32(a0, b1, acc[0][1], 0, 0, 0);
      acc[1][0] = __builtin_amdgcn_mfma_f32_32x32x2f32(a1, b0, acc[1][0], 0, 0, 0);
      acc[1][1] = __builtin_amdgcn_mfma_f32_32x32x2f32(a1, b1, acc[1][1], 0, 0, 0);
    }
    buf ^= 1;
  }

  // Accumulator layout of v_mfma_f32_32x32x2_f32: lane l, register r holds
  // row 8*(r/4) + 4*(l/32) + r%4 and column l%32 of the 32 x 32 block.
  float* C = pi ? P1.C : P0.C;
  const int64_t ldc = pi ? P1.ldc : P0.ldc;
  const float* bias = pi ? P1.bias : P0.bias;
  const int relu = pi ? P1.relu : P0.relu;
  float* part = pi ? g.part[1] : g.part[0];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int col = n0 + wn * 64 + j * 32 + lr;
      if (col >= N) continue;
      const float bc = (g.splits == 1 && bias) ? bias[col] : 0.f;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int row = m0 + wm * 64 + i * 32 + (r >> 2) * 8 + lk * 4 + (r & 3);
        if (row < M) {
          float v = acc[i][j][r];
          if (g.splits > 1) {
            part[((int64_t)split * M + row) * N + col] = v;
          } else {
            v += bc;
            if (relu) v = fmaxf(v, 0.f);
            C[(int64_t)row * ldc + col] = v;
          }
        }
      }
    }
}

// Sum of the split-K partial tiles in split order, then bias and ReLU.
__global__ __launch_bounds__(256) void gemm_splitk_reduce_kernel(GemmKArgs g) {
  const int pi = blockIdx.y;
  const GemmProblem& P0 = g.p[0];
  const GemmProblem& P1 = g.p[1];
  const int M = pi ? P1.M : P0.M;
  const int N = pi ? P1.N : P0.N;
  float* C = pi ? P1.C : P0.C;
  const int64_t ldc = pi ? P1.ldc : P0.ldc;
  const float* bias = pi ? P1.bias : P0.bias;
  const int relu = pi ? P1.relu : P0.relu;
  const float* part = pi ? g.part[1] : g.part[0];
  const int64_t total = (int64_t)M * N;
  for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < total;
       e += (int64_t)gridDim.x * blockDim.x) {
    float v = 0.f;
    for (int s = 0; s < g.splits; ++s) v += part[(int64_t)s * total + e];
    const int row = (int)(e / N), col = (int)(e % N);
    if (bias) v += bias[col];
    if (relu) v = fmaxf(v, 0.f);
    C[(int64_t)row * ldc + col] = v;
  }
}

// ------------------------------------------------------------------ host

static int problem_ktiles(const GemmProblem& p, int* kt0) {
  int k0 = (int)ceil_div(p.seg[0].K, BK);
  int k1 = p.nseg > 1 ? (int)ceil_div(p.seg[1].K, BK) : 0;
  if (kt0) *kt0 = k0;
  return k0 + k1;
}

static int choose_splits(const GemmBatch& b) {
  int tiles = 0, kt = 0;
  for (int i = 0; i < b.nprob; ++i) {
    const GemmProblem& p = b.p[i];
    tiles += (int)(ceil_div(p.M, BM) * ceil_div(p.N, BN));
    kt = std::max(kt, problem_ktiles(p, nullptr));
  }
  if (tiles >= 256 || tiles == 0) return 1;
  int s = (int)ceil_div(512, tiles);
  s = std::min(s, std::max(1, kt / 4));
  return std::max(1, std::min(s, 32));
}

size_t gemm_workspace_bytes(const GemmBatch& b) {
  const int s = choose_splits(b);
  if (s <= 1) return 0;
  size_t bytes = 0;
  for (int i = 0; i < b.nprob; ++i)
    bytes += round_up((size_t)s * b.p[i].M * b.p[i].N * 4, 256);
  return bytes;
}

double gemm_flops(const GemmBatch& b) {
  double f = 0;
  for (int i = 0; i < b.nprob; ++i) {
    const GemmProblem& p = b.p[i];
    for (int s = 0; s < p.nseg; ++s) f += 2.0 * p.M * p.N * (double)p.seg[s].K;
  }
  return f;
}

hipError_t gemm_launch(const GemmBatch& b, void* workspace, size_t ws_bytes,
                       hipStream_t s) {
  GemmKArgs g;
  memset(&g, 0, sizeof(g));
  g.nprob = b.nprob;
  g.splits = choose_splits(b);
  int tiles = 0;
  bool va = true, vb = true;
  char* ws = static_cast<char*>(workspace);
  for (int i = 0; i < b.nprob; ++i) {
    g.p[i] = b.p[i];
    if (g.p[i].nseg < 2) {
      g.p[i].seg[1] = g.p[i].seg[0];
      g.p[i].seg[1].K = 0;
    }
    const GemmProblem& p = g.p[i];
    g.tiles_m[i] = (int)ceil_div(p.M, BM);
    g.tile_start[i] = tiles;
    tiles += g.tiles_m[i] * (int)ceil_div(p.N, BN);
    g.ktiles[i] = problem_ktiles(p, &g.ktiles0[i]);
    for (int k = 0; k < p.nseg; ++k) {
      va = va && vec4_ok(p.seg[k].A, p.seg[k].lda);
      vb = vb && vec4_ok(p.seg[k].B, p.seg[k].ldb);
    }
    if (g.splits > 1) {
      g.part[i] = reinterpret_cast<float*>(ws);
      ws += round_up((size_t)g.splits * p.M * p.N * 4, 256);
    }
  }
  if (g.splits > 1 && (size_t)(ws - static_cast<char*>(workspace)) > ws_bytes)
    return hipErrorInvalidValue;
  g.total_tiles = tiles;
  g.vec_a = va;
  g.vec_b = vb;
  if (tiles == 0) return hipSuccess;
  const unsigned grid = (unsigned)tiles * (unsigned)g.splits;
  const int kid = b.trans_a ? (b.trans_b ? GNN_K_GEMM_TT : GNN_K_GEMM_TN)
                            : (b.trans_b ? GNN_K_GEMM_NT : GNN_K_GEMM_NN);
  timer_begin(kid, s);
  if (!b.trans_a && !b.trans_b)
    gemm_f32_kernel<false, false><<<grid, 256, 0, s>>>(g);
  else if (b.trans_a && !b.trans_b)
    gemm_f32_kernel<true, false><<<grid, 256, 0, s>>>(g);
  else if (!b.trans_a && b.trans_b)
    gemm_f32_kernel<false, true><<<grid, 256, 0, s>>>(g);
  else
    gemm_f32_kernel<true, true><<<grid, 256, 0, s>>>(g);
  timer_end(kid, gemm_flops(b), s);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || g.splits <= 1) return e;
  int64_t maxmn = 0;
  for (int i = 0; i < b.nprob; ++i)
    maxmn = std::max<int64_t>(maxmn, (int64_t)b.p[i].M * b.p[i].N);
  const unsigned rgrid = (unsigned)std::min<int64_t>(ceil_div(maxmn, 256), 4096);
  dim3 grid2(rgrid > 0 ? rgrid : 1, b.nprob);
  timer_begin(GNN_K_GEMM_REDUCE, s);
  gemm_splitk_reduce_kernel<<<grid2, 256, 0, s>>>(g);
  timer_end(GNN_K_GEMM_REDUCE, 0.0, s);
  return hipGetLastError();
}

}  // namespace gnnprop
