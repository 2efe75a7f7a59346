// Dense weight transformation on the gfx950 matrix cores (the second of the
// three kernels of Section 5.1).
//
// C = sum_s op(A_s) op(B_s) (+ bias, ReLU), fp32 in and out.  Products, by
// GemmBatch::mode:
//   split (default, gemm_split_kernel further down): every fp32 operand
//     value split exactly into bf16 hi + mid + lo as it is staged into LDS;
//     the six piece products down to 2^-16 of hi x hi run on
//     v_mfma_f32_32x32x16_bf16 with fp32 accumulation (the bf16x6 scheme of
//     Henry, Tang and Heinecke, 2019).  Six 16-deep bf16 MFMAs take 192
//     cycles against 512 for the eight 2-deep fp32 MFMAs that cover the same
//     16 k, and the result is as accurate (measured against fp64);
//   fp32 (gemm_f32_kernel): v_mfma_f32_32x32x2_f32, described below;
//   bf16 (gemm_bf16_kernel): operands rounded to bf16, one product.
//
// Tiling.  A block of 256 threads (4 wavefronts in 2 x 2) computes a
// 128 x 128 output tile; each wavefront holds a 64 x 64 sub-tile as 2 x 2
// MFMA accumulators (64 accumulator registers per lane).  K advances in
// 32-deep slices staged through double-buffered LDS with one barrier per
// slice.  For interior tiles over full slices the loop is a three-stage
// software pipeline in one basic block: while the matrix cores consume slice
// k from one LDS stage, slice k+1 goes from registers into the other stage
// and the global loads of slice k+2 are issued, interleaved with the MFMAs.
// Edge tiles and partial slices take a guarded path with one slice of
// register prefetch.
//
// LDS layouts follow the operand's storage so that every global float4 lands
// in LDS as one float4 (no transposition on the way in):
//   K-contiguous operand (A row-major M x K, or B stored N x K): [x][k]
//     rows of 32 + 4 floats; each lane fetches its MFMA fragments for 16
//     consecutive k with four 128-bit reads;
//   X-contiguous operand (A stored K x M, or B row-major K x N): [k][x]
//     rows of 128 + 32 floats; one 32-bit read per MFMA.
// The MFMA contracts over k in any order, so within a slice the lane half
// h = lane / 32 takes k = 16 h + s at step s (s = 0..15), which is what
// lets a K-contiguous fragment be read as consecutive floats.  X-contiguous
// rows are stored in the order (k mod 16) * 2 + k / 16 so that the two lane
// halves of a step read adjacent rows (different LDS banks).
//
// Work split (gemm_shape).  One block per tile when the tiles fill the 512
// resident slots (2 per CU), or come to about one per CU over a short K;
// split-K (one (tile, K range) per block) for few tiles over a long K
// (weight gradients, K = n); otherwise stream-K: the launch's tiles x
// K-slices cut into 512 equal, contiguous ranges, one per block (f_in = 602
// input gradients).  A block writes a tile it covers completely straight to
// C with the fused epilogue; a tile shared by several blocks gets one
// partial tile per block, and a second kernel adds them in block order
// (deterministic) before the epilogue, so no atomics are involved.
// Blocks are numbered so that each XCD (blocks are dispatched round-robin
// over the 8 XCDs) works on a contiguous range of iterations: the tiles of a
// row band (same A rows) or the same K range stay in one XCD's L2.
#include "internal.hpp"

namespace gnnprop {

typedef float floatx16 __attribute__((ext_vector_type(16)));

constexpr int BM = 128, BN = 128, BK = 32;
constexpr int KC_STRIDE = BK + 4;   // floats per [x][k] row
constexpr int XC_STRIDE = 128 + 32; // floats per [k][x] row
constexpr int KC_FLOATS = 128 * KC_STRIDE;
constexpr int XC_FLOATS = BK * XC_STRIDE;
constexpr int NUM_XCD = 8;
constexpr int NUM_CU = 256;
constexpr int MAX_BLOCKS = 2 * NUM_CU;  // 2 resident blocks on each CU

struct GemmKArgs {
  GemmProblem p[2];
  int32_t nprob;
  int32_t M;           // shared by the problems of a launch
  int32_t tiles_m;
  int32_t tiles_n0;    // column tiles of problem 0
  int32_t tiles_n;     // column tiles of both problems
  int32_t tiles;       // tiles_m * tiles_n
  int32_t ktiles;      // K slices per tile (same for every problem)
  int32_t ktiles0[2];  // K slices of segment 0, per problem
  int64_t iters;       // tiles * ktiles
  int32_t nblocks;     // P
  int32_t splits;      // > 1: split-K mode, one (tile, K range) per block
  float* part;         // partial tiles (2 per block stream-K, 1 split-K)
  int32_t vec_a, vec_b;
  int32_t vec_c[2];    // C (and mask, bias) of problem i take float4 accesses
};

__device__ inline float4 ld4(const float* p) {
  return *reinterpret_cast<const float4*>(p);
}
__device__ inline float comp(const float4& v, int u) {
  return u == 0 ? v.x : u == 1 ? v.y : u == 2 ? v.z : v.w;
}

// Element (r, c..c+3) of a row-major R x C matrix with row stride ld; zeros
// outside the matrix.
__device__ inline float4 load4(const float* base, int64_t ld, int r, int c,
                               int R, int C, bool vec) {
  float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
  if (r < R && c < C) {
    const float* p = base + (int64_t)r * ld + c;
    if (vec && c + 3 < C) {
      v = ld4(p);
    } else {
      v.x = p[0];
      if (c + 1 < C) v.y = p[1];
      if (c + 2 < C) v.z = p[2];
      if (c + 3 < C) v.w = p[3];
    }
  }
  return v;
}

// Element (r, c..c+1) of a row-major R x C matrix, zeros outside; `vec`
// (8-byte aligned rows, c even) allows one 8-byte load.
__device__ inline float2 load2(const float* base, int64_t ld, int r, int c, int R, int C,
                               bool vec) {
  float2 v = make_float2(0.f, 0.f);
  if (r < R && c < C) {
    const float* p = base + (int64_t)r * ld + c;
    if (vec && c + 1 < C) {
      v = *reinterpret_cast<const float2*>(p);
    } else {
      v.x = p[0];
      if (c + 1 < C) v.y = p[1];
    }
  }
  return v;
}

__device__ inline int64_t block_lo(int b, int64_t iters, int nblocks) {
  return (int64_t)b * iters / nblocks;
}
// The block whose range contains iteration x.
__device__ inline int block_of(int64_t x, int64_t iters, int nblocks) {
  return (int)(((x + 1) * nblocks - 1) / iters);
}

// Logical block of physical block b: XCD x (= b mod 8) gets a contiguous
// range of logical blocks.
__device__ inline int logical_block(int b, int nblocks) {
  const int x = b % NUM_XCD, c = b / NUM_XCD;
  const int base = nblocks / NUM_XCD, rem = nblocks % NUM_XCD;
  return x * base + min(x, rem) + c;
}

// A tile's origin (m0, n0) and the first row / column it owns (r0, c0).
// The last tile of a ragged dimension of at least one tile is moved back
// to end at the matrix edge (m0 = M - BM), so that it runs the unguarded
// pipeline like every other tile; it recomputes the rows (columns) below
// r0 (c0), which belong to its neighbour, and writes only its own.
struct TileInfo {
  int pi, m0, n0, r0, c0;
};

__device__ inline TileInfo tile_info(const GemmKArgs& g, int t) {
  TileInfo ti;
  const int tm = t / g.tiles_n, j = t % g.tiles_n;
  ti.pi = (g.nprob > 1 && j >= g.tiles_n0) ? 1 : 0;
  ti.r0 = tm * BM;
  ti.c0 = (ti.pi ? j - g.tiles_n0 : j) * BN;
  const int N = ti.pi ? g.p[1].N : g.p[0].N;
  ti.m0 = (g.M >= BM && ti.r0 + BM > g.M) ? g.M - BM : ti.r0;
  ti.n0 = (N >= BN && ti.c0 + BN > N) ? N - BN : ti.c0;
  return ti;
}

// Writes a wavefront's 64 x 64 accumulators (layout of the 32 x 32 MFMAs:
// lane l, register r holds row 8*(r/4) + 4*(l/32) + r%4 and column l%32 of a
// block): straight to C with bias, ReLU and mask when the block covered the
// whole K range, else to its partial tile.  Interior tiles take a path
// without per-element guards, so the mask loads go out sixteen at a time.
//
// Whole interior tiles whose C (and mask, bias) take float4 accesses go
// through LDS instead: each wavefront writes one 32 x 32 block at a time
// into its own region (rows of 40 floats: the two lane halves' rows land 32
// banks apart), reads it back as float4 along rows and stores 8 rows of
// 128 bytes per instruction, with the same bias, ReLU and mask.  `lds0` and
// `lds1` are two LDS arrays of at least 2 x 1280 floats that no wavefront
// reads any more (the K loop ended with a barrier); the path ends with a
// barrier, so the next tile may write them.  The condition is uniform over
// the block.
constexpr int EPI_ROW = 40;
constexpr int EPI_REGION = 32 * EPI_ROW;

// NJ: 32-column blocks per wavefront (2: 4 wavefronts of 64 x 64; 1: 8 of
// 64 x 32); WPH wavefronts share each of lds0 and lds1.
template <int NJ = 2, int WPH = 2>
__device__ inline void store_acc(const GemmProblem& P, const TileInfo& ti,
                                 int M, const floatx16 (&acc)[2][NJ],
                                 bool whole, float* part, int wm, int wn,
                                 int lr, int lh, bool vec_c, float* lds0,
                                 float* lds1) {
  const int N = P.N;
  // moved-back tiles take the guarded path, which skips what they do not own
  const bool interior = ti.m0 + BM <= M && ti.n0 + BN <= N && ti.m0 == ti.r0 &&
                        ti.n0 == ti.c0;
  if (whole && interior && vec_c) {
    const int wave = 2 * wn + wm, lane = lh * 32 + lr;
    float* L = (wave < WPH ? lds0 : lds1) + (wave % WPH) * EPI_REGION;
    const int rr = lane >> 3, c4 = 4 * (lane & 7);
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int j = 0; j < NJ; ++j) {
#pragma unroll
        for (int r = 0; r < 16; ++r)
          L[(8 * (r >> 2) + 4 * lh + (r & 3)) * EPI_ROW + lr] = acc[i][j][r];
        const int row0 = ti.m0 + wm * 64 + i * 32,
                  col = ti.n0 + wn * 32 * NJ + j * 32 + c4;
        const float4 bc = P.bias ? ld4(P.bias + col) : make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int row = row0 + rr + 8 * q;
          float4 v = ld4(&L[(rr + 8 * q) * EPI_ROW + c4]);
          v.x += bc.x; v.y += bc.y; v.z += bc.z; v.w += bc.w;
          if (P.relu) {
            v.x = fmaxf(v.x, 0.f); v.y = fmaxf(v.y, 0.f);
            v.z = fmaxf(v.z, 0.f); v.w = fmaxf(v.w, 0.f);
          }
          if (P.mask) {
            const float4 m = ld4(P.mask + (int64_t)row * P.ld_mask + col);
            if (!(m.x > 0.f)) v.x = 0.f;
            if (!(m.y > 0.f)) v.y = 0.f;
            if (!(m.z > 0.f)) v.z = 0.f;
            if (!(m.w > 0.f)) v.w = 0.f;
          }
          *reinterpret_cast<float4*>(P.C + (int64_t)row * P.ldc + col) = v;
        }
      }
    __syncthreads();
    return;
  }
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < NJ; ++j) {
      const int cl = wn * 32 * NJ + j * 32 + lr;
      const int col = ti.n0 + cl;
      const int rl0 = wm * 64 + i * 32 + lh * 4;
      if (!whole) {
#pragma unroll
        for (int r = 0; r < 16; ++r)
          part[(rl0 + (r >> 2) * 8 + (r & 3)) * BN + cl] = acc[i][j][r];
      } else if (interior) {
        const float bc = P.bias ? P.bias[col] : 0.f;
        float mv[16];
        if (P.mask) {
#pragma unroll
          for (int r = 0; r < 16; ++r)
            mv[r] = P.mask[(int64_t)(ti.m0 + rl0 + (r >> 2) * 8 + (r & 3)) * P.ld_mask + col];
        }
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int row = ti.m0 + rl0 + (r >> 2) * 8 + (r & 3);
          float v = acc[i][j][r] + bc;
          if (P.relu) v = fmaxf(v, 0.f);
          if (P.mask && !(mv[r] > 0.f)) v = 0.f;
          P.C[(int64_t)row * P.ldc + col] = v;
        }
      } else {
        const float bc = (P.bias && col < N) ? P.bias[col] : 0.f;
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int row = ti.m0 + rl0 + (r >> 2) * 8 + (r & 3);
          if (row < M && col < N && row >= ti.r0 && col >= ti.c0) {
            float v = acc[i][j][r] + bc;
            if (P.relu) v = fmaxf(v, 0.f);
            if (P.mask && !(P.mask[(int64_t)row * P.ld_mask + col] > 0.f)) v = 0.f;
            P.C[(int64_t)row * P.ldc + col] = v;
          }
        }
      }
    }
}

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

// Tiles shared by several blocks: add the blocks' partial tiles in block
// order, then bias and ReLU.  Chunk c of tile t is 1024 elements, four
// consecutive columns per thread of a 256-thread block.  Run by
// gemm_fixup_kernel, or by extra blocks at the end of the next GEMM launch
// on the stream (which reads the partials the earlier launch wrote).
constexpr int FIX_CHUNKS = BM * BN / 1024;

__device__ inline void fixup_chunk(const GemmKArgs& g, int t, int chunk) {
  const int64_t first = (int64_t)t * g.ktiles, last = first + g.ktiles - 1;
  int b0 = 0, b1 = 0;
  if (g.splits <= 1) {
    b0 = block_of(first, g.iters, g.nblocks);
    b1 = block_of(last, g.iters, g.nblocks);
    if (b0 == b1) return;  // written directly by its only block
  }
  const TileInfo ti = tile_info(g, t);
  const GemmProblem& P = ti.pi ? g.p[1] : g.p[0];
  const int e = chunk * 1024 + threadIdx.x * 4;
  const int rl = e / BN, cl = e % BN;
  const int row = ti.m0 + rl, col = ti.n0 + cl;
  if (row >= g.M || col >= P.N || row < ti.r0) return;
  float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
  if (g.splits > 1) {
    const float* src = g.part + (int64_t)t * (BM * BN) + e;
    const int64_t st = (int64_t)g.tiles * (BM * BN);
    int sp = 0;
    for (; sp + 4 <= g.splits; sp += 4) {  // four partials in flight, in order
      float4 p[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) p[u] = ld4(src + (sp + u) * st);
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        v.x += p[u].x;
        v.y += p[u].y;
        v.z += p[u].z;
        v.w += p[u].w;
      }
    }
    for (; sp < g.splits; ++sp) {
      const float4 p = ld4(src + sp * st);
      v.x += p.x;
      v.y += p.y;
      v.z += p.z;
      v.w += p.w;
    }
  } else {
    for (int b = b0; b <= b1; ++b) {
      // the tile is block b's first tile iff b's range starts inside it
      const int slot = block_lo(b, g.iters, g.nblocks) >= first ? 0 : 1;
      const float4 p = ld4(g.part + ((int64_t)b * 2 + slot) * (BM * BN) + e);
      v.x += p.x;
      v.y += p.y;
      v.z += p.z;
      v.w += p.w;
    }
  }
  float o[4] = {v.x, v.y, v.z, v.w};
  float* dst = P.C + (int64_t)row * P.ldc + col;
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    if (col + u >= P.N) break;
    if (col + u < ti.c0) continue;  // its neighbour's column
    float x = o[u];
    if (P.bias) x += P.bias[col + u];
    if (P.relu) x = fmaxf(x, 0.f);
    if (P.mask && !(P.mask[(int64_t)row * P.ld_mask + col + u] > 0.f)) x = 0.f;
    dst[u] = x;
  }
}

__global__ __launch_bounds__(256) void gemm_fixup_kernel(GemmKArgs g) {
  fixup_chunk(g, blockIdx.x, blockIdx.y);
}

// Blocks past the GEMM's own run the chunks of a reduction left by the
// previous launch (`fx`, fx.tiles x FIX_CHUNKS of them); true for those.
__device__ inline bool run_pending_fixup(const GemmKArgs& g, const GemmKArgs& fx) {
  if ((int)blockIdx.x < g.nblocks) return false;
  if (threadIdx.x >= 256) return true;  // a chunk takes 256 threads
  const int f = (int)blockIdx.x - g.nblocks;
  fixup_chunk(fx, f / FIX_CHUNKS, f % FIX_CHUNKS);
  return true;
}


template <bool AT, bool BT>
__global__ __launch_bounds__(256, 2) void gemm_f32_kernel(GemmKArgs g, GemmKArgs fx) {
  if (run_pending_fixup(g, fx)) return;
  constexpr bool A_KC = !AT;  // A row-major M x K: k contiguous
  constexpr bool B_KC = BT;   // B stored N x K: k contiguous
  constexpr int A_FLOATS = A_KC ? KC_FLOATS : XC_FLOATS;
  constexpr int B_FLOATS = B_KC ? KC_FLOATS : XC_FLOATS;
  // Two LDS stages as separate arrays, so that the compiler sees that the
  // stores into one stage never alias the fragment reads of the other.
  __shared__ __attribute__((aligned(16))) float As0[A_FLOATS];
  __shared__ __attribute__((aligned(16))) float As1[A_FLOATS];
  __shared__ __attribute__((aligned(16))) float Bs0[B_FLOATS];
  __shared__ __attribute__((aligned(16))) float Bs1[B_FLOATS];
  static_assert(A_FLOATS >= 2 * EPI_REGION && B_FLOATS >= 2 * EPI_REGION, "epilogue regions");

  const int tid = threadIdx.x;
  const int wave = tid >> 6, lane = tid & 63;
  const int wm = wave & 1, wn = wave >> 1;
  const int lr = lane & 31, lh = lane >> 5;
  const bool va = g.vec_a != 0, vb = g.vec_b != 0;
  const int M = g.M;

  const int lb = logical_block(blockIdx.x, g.nblocks);
  int64_t lo, hi;
  if (g.splits > 1) {  // block lb = split * tiles + tile
    const int sp = lb / g.tiles, t = lb % g.tiles;
    lo = (int64_t)t * g.ktiles + (int64_t)sp * g.ktiles / g.splits;
    hi = (int64_t)t * g.ktiles + (int64_t)(sp + 1) * g.ktiles / g.splits;
  } else {
    lo = block_lo(lb, g.iters, g.nblocks);
    hi = block_lo(lb + 1, g.iters, g.nblocks);
  }

  int seg = 0;
  for (int64_t it = lo; it < hi; ++seg) {
    const int t = (int)(it / g.ktiles);
    const int kbeg = (int)(it - (int64_t)t * g.ktiles);
    const int kend = (int)min<int64_t>(g.ktiles, hi - (int64_t)t * g.ktiles);
    it = (int64_t)t * g.ktiles + kend;
    const TileInfo ti = tile_info(g, t);
    const GemmProblem& P = ti.pi ? g.p[1] : g.p[0];
    const int N = P.N;
    const int m0 = ti.m0, n0 = ti.n0;
    // Segment parameters, read once per tile (kept in scalar registers).
    const int kt0 = ti.pi ? g.ktiles0[1] : g.ktiles0[0];
    const float* const A0p = P.seg[0].A;
    const float* const A1p = P.seg[1].A;
    const float* const B0p = P.seg[0].B;
    const float* const B1p = P.seg[1].B;
    const int64_t lda0 = P.seg[0].lda, lda1 = P.seg[1].lda;
    const int64_t ldb0 = P.seg[0].ldb, ldb1 = P.seg[1].ldb;
    const int K0 = P.seg[0].K, K1 = P.seg[1].K;
    const bool a_in = va && m0 + BM <= M;  // no row/column guard needed
    const bool b_in = vb && n0 + BN <= N;
    // This thread's place in a slice: KC operands own (row x, 4 k),
    // XC operands own (row k, 4 consecutive m or n).
    const int ax = A_KC ? (tid >> 3) : (tid >> 5);
    const int ay = A_KC ? 4 * (tid & 7) : 4 * (tid & 31);
    const int bx = B_KC ? (tid >> 3) : (tid >> 5);
    const int by = B_KC ? 4 * (tid & 7) : 4 * (tid & 31);
    constexpr int ASTEP = A_KC ? 32 : 8;
    constexpr int BSTEP = B_KC ? 32 : 8;

    float4 ra[4], rb[4];
    // Any slice: guarded loads, zeros outside the operands.
    auto load_slice = [&](int ks) {
      const bool s1 = ks >= kt0;
      const float* A = s1 ? A1p : A0p;
      const float* B = s1 ? B1p : B0p;
      const int64_t lda = s1 ? lda1 : lda0;
      const int64_t ldb = s1 ? ldb1 : ldb0;
      const int K = s1 ? K1 : K0;
      const int k0 = (s1 ? ks - kt0 : ks) * BK;
      const bool fk = k0 + BK <= K;
      if (a_in && fk) {
        const float* p0 = A_KC ? A + (int64_t)(m0 + ax) * lda + (k0 + ay)
                               : A + (int64_t)(k0 + ax) * lda + (m0 + ay);
        const int64_t st = ASTEP * lda;
#pragma unroll
        for (int p = 0; p < 4; ++p) ra[p] = ld4(p0 + p * st);
      } else {
#pragma unroll
        for (int p = 0; p < 4; ++p)
          ra[p] = A_KC ? load4(A, lda, m0 + ax + ASTEP * p, k0 + ay, M, K, va)
                       : load4(A, lda, k0 + ax + ASTEP * p, m0 + ay, K, M, va);
      }
      if (b_in && fk) {
        const float* p0 = B_KC ? B + (int64_t)(n0 + bx) * ldb + (k0 + by)
                               : B + (int64_t)(k0 + bx) * ldb + (n0 + by);
        const int64_t st = BSTEP * ldb;
#pragma unroll
        for (int p = 0; p < 4; ++p) rb[p] = ld4(p0 + p * st);
      } else {
#pragma unroll
        for (int p = 0; p < 4; ++p)
          rb[p] = B_KC ? load4(B, ldb, n0 + bx + BSTEP * p, k0 + by, N, K, vb)
                       : load4(B, ldb, k0 + bx + BSTEP * p, n0 + by, K, N, vb);
      }
    };
    // A full slice of an interior tile: no guards, no branches.
    auto load_full = [&](int ks) {
      const bool s1 = ks >= kt0;
      const float* A = s1 ? A1p : A0p;
      const float* B = s1 ? B1p : B0p;
      const int64_t lda = s1 ? lda1 : lda0;
      const int64_t ldb = s1 ? ldb1 : ldb0;
      const int k0 = (s1 ? ks - kt0 : ks) * BK;
      const float* pa = A_KC ? A + (int64_t)(m0 + ax) * lda + (k0 + ay)
                             : A + (int64_t)(k0 + ax) * lda + (m0 + ay);
      const float* pb = B_KC ? B + (int64_t)(n0 + bx) * ldb + (k0 + by)
                             : B + (int64_t)(k0 + bx) * ldb + (n0 + by);
      const int64_t sa = ASTEP * lda, sb = BSTEP * ldb;
#pragma unroll
      for (int p = 0; p < 4; ++p) {
        ra[p] = ld4(pa + p * sa);
        rb[p] = ld4(pb + p * sb);
      }
    };
    // LDS offsets (floats) of this thread's slice stores.
    auto sto_off = [&](bool kc, int x, int y, int p, int step) {
      if (kc) return (x + step * p) * KC_STRIDE + y;
      const int kk = x + step * p;
      return (((kk & 15) << 1) | (kk >> 4)) * XC_STRIDE + y;
    };
    auto store_slice = [&](float* as, float* bs) {
#pragma unroll
      for (int p = 0; p < 4; ++p) {
        *reinterpret_cast<float4*>(&as[sto_off(A_KC, ax, ay, p, ASTEP)]) = ra[p];
        *reinterpret_cast<float4*>(&bs[sto_off(B_KC, bx, by, p, BSTEP)]) = rb[p];
      }
    };

    floatx16 acc[2][2];
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int j = 0; j < 2; ++j)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

    // Fragment reads.  Step s of a slice uses k = 16 * lh + s.  KC operands
    // come in float4 groups of 4 steps (q = s / 4); XC operands one float per
    // step from the stored row 2 s + lh.
    const int a_kc_base = (wm * 64 + lr) * KC_STRIDE + lh * 16;
    const int b_kc_base = (wn * 64 + lr) * KC_STRIDE + lh * 16;
    const int a_xc_base = lh * XC_STRIDE + wm * 64 + lr;
    const int b_xc_base = lh * XC_STRIDE + wn * 64 + lr;

    auto compute = [&](const float* as, const float* bs) {
      // Operands of step s are fetched one step (XC) or one group (KC)
      // ahead of the MFMAs that consume them.
      float4 af[2], bf[2], afn[2], bfn[2];
      float ax_[2], bx_[2], axn[2], bxn[2];
#pragma unroll
      for (int i = 0; i < 2; ++i) {
        if (A_KC) afn[i] = ld4(as + a_kc_base + i * 32 * KC_STRIDE);
        else axn[i] = as[a_xc_base + i * 32];
        if (B_KC) bfn[i] = ld4(bs + b_kc_base + i * 32 * KC_STRIDE);
        else bxn[i] = bs[b_xc_base + i * 32];
      }
#pragma unroll
      for (int st = 0; st < BK / 2; ++st) {
        const int u = st & 3;
        if (u == 0) {
#pragma unroll
          for (int i = 0; i < 2; ++i) {
            af[i] = afn[i];
            bf[i] = bfn[i];
          }
          if (st + 4 < BK / 2) {
#pragma unroll
            for (int i = 0; i < 2; ++i) {
              if (A_KC) afn[i] = ld4(as + a_kc_base + i * 32 * KC_STRIDE + st + 4);
              if (B_KC) bfn[i] = ld4(bs + b_kc_base + i * 32 * KC_STRIDE + st + 4);
            }
          }
        }
#pragma unroll
        for (int i = 0; i < 2; ++i) {
          ax_[i] = axn[i];
          bx_[i] = bxn[i];
        }
        if (st + 1 < BK / 2) {
#pragma unroll
          for (int i = 0; i < 2; ++i) {
            if (!A_KC) axn[i] = as[a_xc_base + 2 * (st + 1) * XC_STRIDE + i * 32];
            if (!B_KC) bxn[i] = bs[b_xc_base + 2 * (st + 1) * XC_STRIDE + i * 32];
          }
        }
        float a[2], b[2];
#pragma unroll
        for (int i = 0; i < 2; ++i) {
          a[i] = A_KC ? comp(af[i], u) : ax_[i];
          b[i] = B_KC ? comp(bf[i], u) : bx_[i];
        }
        acc[0][0] = __builtin_amdgcn_mfma_f32_32x32x2f32(a[0], b[0], acc[0][0], 0, 0, 0);
        acc[0][1] = __builtin_amdgcn_mfma_f32_32x32x2f32(a[0], b[1], acc[0][1], 0, 0, 0);
        acc[1][0] = __builtin_amdgcn_mfma_f32_32x32x2f32(a[1], b[0], acc[1][0], 0, 0, 0);
        acc[1][1] = __builtin_amdgcn_mfma_f32_32x32x2f32(a[1], b[1], acc[1][1], 0, 0, 0);
      }
    };

    // One pipelined step over a full slice: store the next slice (already
    // in registers) into the other stage, issue the global loads of the
    // slice after it, compute on the current stage, then one barrier.  The
    // three are one basic block, so the MFMAs interleave with the memory
    // operations.  Near the end of the range the load repeats the last
    // slice and the store fills the idle stage; neither is read again.
    auto step = [&](const float* as, const float* bs, float* as_n, float* bs_n,
                    int kl) {
      // the second-round block of the CU first (see gemm_split_kernel)
      if (blockIdx.x >= NUM_CU)
        __builtin_amdgcn_s_setprio(1);
      else
        __builtin_amdgcn_s_setprio(0);
      store_slice(as_n, bs_n);
      load_full(kl);
      compute(as, bs);
      // The stores go out with the first eight MFMAs, the loads with the
      // next eight (a whole step ahead of the stores that consume them),
      // and the fragment reads are spread over the rest.
#pragma unroll
      for (int r = 0; r < 8; ++r) {
        __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);  // LDS read
        __builtin_amdgcn_sched_group_barrier(0x200, 1, 0);  // LDS write
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // MFMA
      }
#pragma unroll
      for (int r = 0; r < 8; ++r) {
        __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);  // LDS read
        __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);  // global load
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // MFMA
      }
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);  // LDS read
        __builtin_amdgcn_sched_group_barrier(0x008, 3, 0);  // MFMA
      }
      __syncthreads();
    };

    // Slices [kbeg, kf) are full and the tile is interior: pipelined path.
    // Every section ends with a barrier, so the next one may write either
    // stage.
    int kf = kbeg;
    if (a_in && b_in) {
      const int f0 = K0 / BK, e1 = kt0 + K1 / BK;
      if (kbeg < f0)
        kf = min(kend, f0 == kt0 ? e1 : f0);
      else if (kbeg >= kt0 && kbeg < e1)
        kf = min(kend, e1);
    }
    if (kf > kbeg) {
      load_full(kbeg);
      store_slice(As0, Bs0);
      load_full(min(kbeg + 1, kf - 1));
      __syncthreads();
      for (int k = kbeg; k < kf; k += 2) {
        step(As0, Bs0, As1, Bs1, min(k + 2, kf - 1));
        if (k + 1 >= kf) break;
        step(As1, Bs1, As0, Bs0, min(k + 3, kf - 1));
      }
    }
    // Remaining slices (edge tiles, partial slices): guarded loads, one
    // slice in registers ahead.
    if (kf < kend) {
      int buf = 0;
      load_slice(kf);
      for (int ks = kf; ks < kend; ++ks) {
        float* as = buf ? As1 : As0;
        float* bs = buf ? Bs1 : Bs0;
        store_slice(as, bs);
        __syncthreads();
        if (ks + 1 < kend) load_slice(ks + 1);
        compute(as, bs);
        __builtin_amdgcn_iglp_opt(0);
        buf ^= 1;
      }
      __syncthreads();
    }

    const bool whole = kbeg == 0 && kend == g.ktiles;
    float* part = g.part + (g.splits > 1 ? (int64_t)lb
                                         : (int64_t)lb * 2 + (seg > 0 ? 1 : 0)) *
                               (BM * BN);
    store_acc(P, ti, M, acc, whole, part, wm, wn, lr, lh, g.vec_c[ti.pi] != 0,
              reinterpret_cast<float*>(As0), reinterpret_cast<float*>(Bs0));
  }
}

// --------------------------------------------------------- bf16 variant
//
// Same tiling, work split and epilogue as the fp32 kernel, with operands
// rounded to bf16 (round to nearest even, v_cvt_pk_bf16_f32) as they are
// staged into LDS and fp32 accumulation on v_mfma_f32_32x32x16_bf16.  A
// 32 x 32 x 16 bf16 MFMA takes a sixteenth of the cycles of the fp32 one, so
// a K step here is 64 deep (four MFMA steps, 16 MFMAs per wavefront between
// barriers) to amortise the per-step chain of waits, conversions, LDS
// stores and the barrier.  In MFMA step s (s = 0..3) lane half h supplies
// the 8 values k = 32 h + 8 s + j (j = 0..7); A and B use the same order,
// so the contraction is unchanged.
//   K-contiguous operand: LDS [x][k] rows of 64 + 8 bf16 (36 words); one
//     128-bit read per fragment.
//   X-contiguous operand: LDS rows of k pairs, each word = (k, k+1) of one
//     x as bf16x2; a fragment is 4 words from 4 pair rows.  Pair kp lives
//     in half kp / 16 (pairs of lane half 0, then of lane half 1), row
//     kp mod 16, and the second half starts 32 words past the first's end,
//     so the two lane halves of a read fall on different banks.
// Interior tiles over full K steps run the fp32 kernel's pipeline: store the
// next step (in registers) into the other LDS stage, issue the loads of the
// step after it, compute, one barrier.
constexpr int BK16 = 64;
constexpr int KC16_STRIDE = BK16 / 2 + 4;          // words per [x][k] row
constexpr int XC16_HALF = (BK16 / 4) * 128 + 32;   // words per half (16 pair rows + gap)
constexpr int KC16_WORDS = 128 * KC16_STRIDE;
constexpr int XC16_WORDS = 2 * XC16_HALF;

// LDS word of k pair kp, column x, in the x-contiguous bf16 layout.
__device__ inline int xc16_word(int kp, int x) {
  return (kp >> 4) * XC16_HALF + (kp & 15) * 128 + x;
}

// Operand storage of the bf16 kernel: fp32 values rounded to bf16 as they
// are staged, or bf16 values already (written so by the kernel that
// produced them), moved unchanged.  R holds 4 consecutive elements of one
// row; kc() gives them as the two k-pair words of the [x][k] layout, xc()
// the four (k, k+1) words of rows a (k) and b (k + 1).
template <bool H>
struct Bf16Op;
template <>
struct Bf16Op<false> {
  using E = float;
  using R = float4;
  __device__ static R fast(const float* p) { return ld4(p); }
  __device__ static R guarded(const float* base, int64_t ld, int r, int c, int Rn,
                              int Cn, bool vec) {
    return load4(base, ld, r, c, Rn, Cn, vec);
  }
  __device__ static uint2 kc(R a) { return make_uint2(pack_bf16(a.x, a.y), pack_bf16(a.z, a.w)); }
  __device__ static uint4 xc(R a, R b) {
    return make_uint4(pack_bf16(a.x, b.x), pack_bf16(a.y, b.y), pack_bf16(a.z, b.z),
                      pack_bf16(a.w, b.w));
  }
};
template <>
struct Bf16Op<true> {
  using E = uint16_t;
  using R = uint2;  // elements c, c + 1 in .x (low, high), c + 2, c + 3 in .y
  __device__ static R fast(const uint16_t* p) { return *reinterpret_cast<const uint2*>(p); }
  __device__ static R guarded(const uint16_t* base, int64_t ld, int r, int c, int Rn,
                              int Cn, bool vec) {
    R v = make_uint2(0u, 0u);
    if (r < Rn && c < Cn) {
      const uint16_t* p = base + (int64_t)r * ld + c;
      if (vec && c + 3 < Cn) {
        v = fast(p);
      } else {
        const uint32_t e0 = p[0], e1 = c + 1 < Cn ? p[1] : 0u;
        const uint32_t e2 = c + 2 < Cn ? p[2] : 0u, e3 = c + 3 < Cn ? p[3] : 0u;
        v.x = e0 | (e1 << 16);
        v.y = e2 | (e3 << 16);
      }
    }
    return v;
  }
  __device__ static uint2 kc(R a) { return a; }
  __device__ static uint4 xc(R a, R b) {
    return make_uint4((a.x & 0xffffu) | (b.x << 16), (a.x >> 16) | (b.x & 0xffff0000u),
                      (a.y & 0xffffu) | (b.y << 16), (a.y >> 16) | (b.y & 0xffff0000u));
  }
};

// A16 / B16: that operand is stored as bf16 (GemmBatch::a16 / b16).
template <bool AT, bool BT, bool A16, bool B16>
__global__ __launch_bounds__(256, 2) void gemm_bf16_kernel(GemmKArgs g, GemmKArgs fx) {
  if (run_pending_fixup(g, fx)) return;
  constexpr bool A_KC = !AT;
  constexpr bool B_KC = BT;
  constexpr int A_WORDS = A_KC ? KC16_WORDS : XC16_WORDS;
  constexpr int B_WORDS = B_KC ? KC16_WORDS : XC16_WORDS;
  __shared__ __attribute__((aligned(16))) uint32_t As0[A_WORDS];
  __shared__ __attribute__((aligned(16))) uint32_t As1[A_WORDS];
  __shared__ __attribute__((aligned(16))) uint32_t Bs0[B_WORDS];
  __shared__ __attribute__((aligned(16))) uint32_t Bs1[B_WORDS];
  static_assert(A_WORDS >= 2 * EPI_REGION && B_WORDS >= 2 * EPI_REGION, "epilogue regions");

  const int tid = threadIdx.x;
  const int wave = tid >> 6, lane = tid & 63;
  const int wm = wave & 1, wn = wave >> 1;
  const int lr = lane & 31, lh = lane >> 5;
  const bool va = g.vec_a != 0, vb = g.vec_b != 0;
  const int M = g.M;

  const int lb = logical_block(blockIdx.x, g.nblocks);
  int64_t lo, hi;
  if (g.splits > 1) {
    const int sp = lb / g.tiles, t = lb % g.tiles;
    lo = (int64_t)t * g.ktiles + (int64_t)sp * g.ktiles / g.splits;
    hi = (int64_t)t * g.ktiles + (int64_t)(sp + 1) * g.ktiles / g.splits;
  } else {
    lo = block_lo(lb, g.iters, g.nblocks);
    hi = block_lo(lb + 1, g.iters, g.nblocks);
  }

  int seg = 0;
  for (int64_t it = lo; it < hi; ++seg) {
    const int t = (int)(it / g.ktiles);
    const int kbeg = (int)(it - (int64_t)t * g.ktiles);
    const int kend = (int)min<int64_t>(g.ktiles, hi - (int64_t)t * g.ktiles);
    it = (int64_t)t * g.ktiles + kend;
    const TileInfo ti = tile_info(g, t);
    const GemmProblem& P = ti.pi ? g.p[1] : g.p[0];
    const int N = P.N;
    const int m0 = ti.m0, n0 = ti.n0;
    const int kt0 = ti.pi ? g.ktiles0[1] : g.ktiles0[0];
    using OA = Bf16Op<A16>;
    using OB = Bf16Op<B16>;
    const auto* const A0p = reinterpret_cast<const typename OA::E*>(P.seg[0].A);
    const auto* const A1p = reinterpret_cast<const typename OA::E*>(P.seg[1].A);
    const auto* const B0p = reinterpret_cast<const typename OB::E*>(P.seg[0].B);
    const auto* const B1p = reinterpret_cast<const typename OB::E*>(P.seg[1].B);
    const int64_t lda0 = P.seg[0].lda, lda1 = P.seg[1].lda;
    const int64_t ldb0 = P.seg[0].ldb, ldb1 = P.seg[1].ldb;
    const int K0 = P.seg[0].K, K1 = P.seg[1].K;
    const bool a_in = va && m0 + BM <= M;
    const bool b_in = vb && n0 + BN <= N;
    // KC: thread owns k = 4 (tid & 15) .. + 3 of rows x = (tid >> 4) + 16 q
    // (q = 0..7): 16 lanes read one 256-byte row, a wavefront 4 whole rows
    // per instruction (8 cache lines per KiB).
    // XC: thread owns k pair kp = (tid >> 5) + 8 p and x = 4 (tid & 31) .. + 3.
    const int kx = tid >> 4, ky = 4 * (tid & 15);
    const int xk = tid >> 5, xy = 4 * (tid & 31);

    typename OA::R ra[8];
    typename OB::R rb[8];
    // One operand's K step: (KC) 4 consecutive k of 8 rows, or (XC) rows
    // 2 kp and 2 kp + 1, for p = 0..3 (Op: the operand's storage).
    auto load_op = [&](auto& r, bool kc, const auto* X, int64_t ld, int x0, int X_extent,
                       int k0, int K, bool fast, bool vec) {
      using Op = Bf16Op<sizeof(*X) == 2>;
#pragma unroll
      for (int p = 0; p < 4; ++p) {
        if (kc) {
          const int x = x0 + kx + 32 * p, k = k0 + ky;
          if (fast) {
            const auto* q = X + (int64_t)x * ld + k;
            r[2 * p] = Op::fast(q);
            r[2 * p + 1] = Op::fast(q + 16 * ld);
          } else {
            r[2 * p] = Op::guarded(X, ld, x, k, X_extent, K, vec);
            r[2 * p + 1] = Op::guarded(X, ld, x + 16, k, X_extent, K, vec);
          }
        } else {
          const int k = k0 + 2 * (xk + 8 * p), x = x0 + xy;
          if (fast) {
            const auto* q = X + (int64_t)k * ld + x;
            r[2 * p] = Op::fast(q);
            r[2 * p + 1] = Op::fast(q + ld);
          } else {
            r[2 * p] = Op::guarded(X, ld, k, x, K, X_extent, vec);
            r[2 * p + 1] = Op::guarded(X, ld, k + 1, x, K, X_extent, vec);
          }
        }
      }
    };
    auto load_slice = [&](int ks) {
      const bool s1 = ks >= kt0;
      const int K = s1 ? K1 : K0;
      const int k0 = (s1 ? ks - kt0 : ks) * BK16;
      const bool fk = k0 + BK16 <= K;
      load_op(ra, A_KC, s1 ? A1p : A0p, s1 ? lda1 : lda0, m0, M, k0, K, a_in && fk, va);
      load_op(rb, B_KC, s1 ? B1p : B0p, s1 ? ldb1 : ldb0, n0, N, k0, K, b_in && fk, vb);
    };
    auto store_op = [&](uint32_t* L, const auto& r, bool kc) {
      using Op = Bf16Op<sizeof(r[0]) == 8>;
#pragma unroll
      for (int p = 0; p < 4; ++p) {
        if (kc) {  // 4 consecutive k of rows x and x + 16
          *reinterpret_cast<uint2*>(&L[(kx + 32 * p) * KC16_STRIDE + ky / 2]) = Op::kc(r[2 * p]);
          *reinterpret_cast<uint2*>(&L[(kx + 32 * p + 16) * KC16_STRIDE + ky / 2]) =
              Op::kc(r[2 * p + 1]);
        } else {   // k pair (row 2kp, row 2kp+1) of 4 consecutive x
          *reinterpret_cast<uint4*>(&L[xc16_word(xk + 8 * p, xy)]) =
              Op::xc(r[2 * p], r[2 * p + 1]);
        }
      }
    };

    floatx16 acc[2][2];
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int j = 0; j < 2; ++j)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

    // fragment for block i of an operand at MFMA step s
    auto frag = [&](const uint32_t* L, bool kc, int wbase, int i, int s) {
      uint4 w;
      const int x = wbase + i * 32 + lr;
      if (kc) {
        w = *reinterpret_cast<const uint4*>(&L[x * KC16_STRIDE + 16 * lh + 4 * s]);
      } else {
        // k pairs 16 lh + 4 s + c
        w.x = L[xc16_word(16 * lh + 4 * s + 0, x)];
        w.y = L[xc16_word(16 * lh + 4 * s + 1, x)];
        w.z = L[xc16_word(16 * lh + 4 * s + 2, x)];
        w.w = L[xc16_word(16 * lh + 4 * s + 3, x)];
      }
      return __builtin_bit_cast(bf16x8, w);
    };
    auto compute = [&](const uint32_t* as, const uint32_t* bs) {
#pragma unroll
      for (int st = 0; st < BK16 / 16; ++st) {
        const bf16x8 a0 = frag(as, A_KC, wm * 64, 0, st);
        const bf16x8 a1 = frag(as, A_KC, wm * 64, 1, st);
        const bf16x8 b0 = frag(bs, B_KC, wn * 64, 0, st);
        const bf16x8 b1 = frag(bs, B_KC, wn * 64, 1, st);
        acc[0][0] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a0, b0, acc[0][0], 0, 0, 0);
        acc[0][1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a0, b1, acc[0][1], 0, 0, 0);
        acc[1][0] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a1, b0, acc[1][0], 0, 0, 0);
        acc[1][1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a1, b1, acc[1][1], 0, 0, 0);
        // keep each MFMA step's fragment reads with it (hoisting all four
        // steps' reads needs 64 more registers than two blocks per CU allow)
        __builtin_amdgcn_sched_barrier(0);
      }
    };

    // Steps [kbeg, kf) are full and the tile is interior: pipelined path.
    int kf = kbeg;
    if (a_in && b_in) {
      const int f0 = K0 / BK16, e1 = kt0 + K1 / BK16;
      if (kbeg < f0)
        kf = min(kend, f0 == kt0 ? e1 : f0);
      else if (kbeg >= kt0 && kbeg < e1)
        kf = min(kend, e1);
    }
    if (kf > kbeg) {
      auto load_full = [&](int ks) {
        ks = min(ks, kf - 1);  // past the end: repeat the last step (never read)
        const bool s1 = ks >= kt0;
        const int k0 = (s1 ? ks - kt0 : ks) * BK16;
        load_op(ra, A_KC, s1 ? A1p : A0p, s1 ? lda1 : lda0, m0, M, k0, 0, true, true);
        load_op(rb, B_KC, s1 ? B1p : B0p, s1 ? ldb1 : ldb0, n0, N, k0, 0, true, true);
      };
      auto step = [&](const uint32_t* as, const uint32_t* bs, uint32_t* as_n,
                      uint32_t* bs_n, int kl) {
        // the second-round block of the CU first (see gemm_split_kernel)
        if (blockIdx.x >= NUM_CU)
          __builtin_amdgcn_s_setprio(1);
        else
          __builtin_amdgcn_s_setprio(0);
        store_op(as_n, ra, A_KC);
        store_op(bs_n, rb, B_KC);
        load_full(kl);
        compute(as, bs);
        __syncthreads();
      };
      load_full(kbeg);
      store_op(As0, ra, A_KC);
      store_op(Bs0, rb, B_KC);
      load_full(kbeg + 1);
      __syncthreads();
      for (int k = kbeg; k < kf; k += 2) {
        step(As0, Bs0, As1, Bs1, k + 2);
        if (k + 1 >= kf) break;
        step(As1, Bs1, As0, Bs0, k + 3);
      }
    }

    // Remaining steps (edge tiles, partial K steps): guarded loads, one step
    // in registers ahead.
    if (kf < kend) {
      int buf = 0;
      load_slice(kf);
      for (int ks = kf; ks < kend; ++ks) {
        uint32_t* as = buf ? As1 : As0;
        uint32_t* bs = buf ? Bs1 : Bs0;
        store_op(as, ra, A_KC);
        store_op(bs, rb, B_KC);
        __syncthreads();
        if (ks + 1 < kend) load_slice(ks + 1);
        compute(as, bs);
        buf ^= 1;
      }
      __syncthreads();
    }

    const bool whole = kbeg == 0 && kend == g.ktiles;
    float* part = g.part + (g.splits > 1 ? (int64_t)lb
                                         : (int64_t)lb * 2 + (seg > 0 ? 1 : 0)) *
                               (BM * BN);
    store_acc(P, ti, M, acc, whole, part, wm, wn, lr, lh, g.vec_c[ti.pi] != 0,
              reinterpret_cast<float*>(As0), reinterpret_cast<float*>(Bs0));
  }
}

// ----------------------------------------------- split-product kernel
//
// The default fp32 mode.  Each operand value is split once per block, as it
// is staged into LDS, into bf16 hi + mid + lo (split3 below; exact), kept in
// three LDS planes; the MFMAs read ready pieces, and the split of the next
// stage does not wait for the current stage's products.  K advances 16 deep
// per stage (one MFMA step: 24 MFMAs per wavefront), which keeps two
// double-buffered stages of three planes per operand within half the LDS of
// a CU (two blocks per CU).
// Lane half h supplies k = 8 h + j (j = 0..7) in both operands.
//   K-contiguous operand: plane [x][k] rows of 8 words (k pairs) + 4 words
//     of padding (48 bytes: eight consecutive rows of a 128-bit fragment
//     read fall on distinct banks); a fragment is one 128-bit read.
//   X-contiguous operand: plane rows of k pairs, word (kp, x) = (k 2kp,
//     2kp + 1) of column x; pairs 4..7 start 32 words past the end of pairs
//     0..3 so that the two lane halves of a read use different banks; a
//     fragment is 4 words from 4 pair rows.
constexpr int BKS = 16;
constexpr int KCS_ROW = 12;
constexpr int KCS_PLANE = 128 * KCS_ROW;
constexpr int XCS_HALF = 4 * 128 + 32;
constexpr int XCS_PLANE = 2 * XCS_HALF;

__device__ inline int xcs_word(int kp, int x) {
  return (kp >> 2) * XCS_HALF + (kp & 3) * 128 + x;
}

// Pieces of the pair (x0, x1): hi, mid and lo packed as bf16x2 words with
// x = hi + mid + lo exactly.
__device__ inline void split3(float x0, float x1, uint32_t& h, uint32_t& m,
                              uint32_t& l) {
  // (the empty asm keeps each packed pair as one value: otherwise the
  // compiler converts each half again to take it apart)
  uint32_t a = pack_bf16(x0, x1);
  asm volatile("" : "+v"(a));
  const float r0 = x0 - __uint_as_float(a << 16);
  const float r1 = x1 - __uint_as_float(a & 0xffff0000u);
  uint32_t b = pack_bf16(r0, r1);
  asm volatile("" : "+v"(b));
  const float s0 = r0 - __uint_as_float(b << 16);
  const float s1 = r1 - __uint_as_float(b & 0xffff0000u);
  h = a;
  m = b;
  l = pack_bf16(s0, s1);
}

// BD: B comes pre-split (GemmSeg::Bp, split_b_planes_launch) and each
// wavefront loads its B fragments straight from those planes into registers
// (one 128-bit load per piece and block: the planes are in fragment order,
// so a fragment is 1 KiB of consecutive bytes), one stage ahead of the
// products that use them; only A goes through the split and LDS.
// NW: wavefronts per block.  4: each computes 64 x 64 of the 128 x 128
// tile.  8 (k-contiguous A): each computes 64 x 32, four wavefronts per
// SIMD at two blocks per CU; a thread stages one float4 of a k-contiguous
// operand, or two columns of one k pair of an x-contiguous one, per stage.
template <bool AT, bool BT, bool BD, int NW = 4>
__global__ __launch_bounds__(NW * 64, NW / 2) void gemm_split_kernel(GemmKArgs g, GemmKArgs fx) {
  static_assert(NW == 4 || (NW == 8 && !AT), "8 wavefronts: k-contiguous A");
  constexpr int NJ = NW == 8 ? 1 : 2;  // 32-column blocks per wavefront
  constexpr int AP = 8 / NW;           // 64-row groups of A staged per thread
  if (run_pending_fixup(g, fx)) return;
  constexpr bool A_KC = !AT;
  constexpr bool B_KC = BT;
  constexpr int A_PLANE = A_KC ? KCS_PLANE : XCS_PLANE;
  constexpr int B_PLANE = B_KC ? KCS_PLANE : XCS_PLANE;
  constexpr int B_WORDS = BD ? 4 : 3 * B_PLANE;
  constexpr int A_WORDS =
      3 * A_PLANE > (NW / 2) * EPI_REGION ? 3 * A_PLANE : (NW / 2) * EPI_REGION;
  __shared__ __attribute__((aligned(16))) uint32_t As0[A_WORDS];
  __shared__ __attribute__((aligned(16))) uint32_t As1[A_WORDS];
  __shared__ __attribute__((aligned(16))) uint32_t Bs0[B_WORDS];
  __shared__ __attribute__((aligned(16))) uint32_t Bs1[B_WORDS];
  static_assert(BD || NW == 8 || 3 * B_PLANE >= 2 * EPI_REGION, "epilogue regions");
  // Two blocks share each CU, and the wavefront arbiter favours the older
  // one: a block of the first dispatch round (every CU receives one before
  // any receives a second) ran ahead of its CU-mate by ~16 us over a 64-stage
  // tile, and the later block then finished alone at half occupancy.  The
  // second-round block takes the higher priority instead: for all of its
  // stages when B comes pre-split, for its first 60 % of stages otherwise
  // (the settings that measured fastest; the two then end within ~2 us of
  // each other).  Priority changes timing only, never results.
  const bool second_round = blockIdx.x >= NUM_CU;

  const int tid = threadIdx.x;
  const int wave = tid >> 6, lane = tid & 63;
  const int wm = wave & 1, wn = wave >> 1;
  const int lr = lane & 31, lh = lane >> 5;
  const bool va = g.vec_a != 0, vb = g.vec_b != 0;
  const int M = g.M;

  const int lb = logical_block(blockIdx.x, g.nblocks);
  int64_t lo, hi;
  if (g.splits > 1) {
    const int sp = lb / g.tiles, t = lb % g.tiles;
    lo = (int64_t)t * g.ktiles + (int64_t)sp * g.ktiles / g.splits;
    hi = (int64_t)t * g.ktiles + (int64_t)(sp + 1) * g.ktiles / g.splits;
  } else {
    lo = block_lo(lb, g.iters, g.nblocks);
    hi = block_lo(lb + 1, g.iters, g.nblocks);
  }

  int seg = 0;
  for (int64_t it = lo; it < hi; ++seg) {
    const int t = (int)(it / g.ktiles);
    const int kbeg = (int)(it - (int64_t)t * g.ktiles);
    const int kend = (int)min<int64_t>(g.ktiles, hi - (int64_t)t * g.ktiles);
    it = (int64_t)t * g.ktiles + kend;
    const TileInfo ti = tile_info(g, t);
    const GemmProblem& P = ti.pi ? g.p[1] : g.p[0];
    const int N = P.N;
    const int m0 = ti.m0, n0 = ti.n0;
    const int kt0 = ti.pi ? g.ktiles0[1] : g.ktiles0[0];
    const float* const A0p = P.seg[0].A;
    const float* const A1p = P.seg[1].A;
    const float* const B0p = P.seg[0].B;
    const float* const B1p = P.seg[1].B;
    const int64_t lda0 = P.seg[0].lda, lda1 = P.seg[1].lda;
    const int64_t ldb0 = P.seg[0].ldb, ldb1 = P.seg[1].ldb;
    const int K0 = P.seg[0].K, K1 = P.seg[1].K;
    const uint32_t* const Bq0 = P.seg[0].Bp;
    const uint32_t* const Bq1 = P.seg[1].Bp;
    const int64_t bps0 = P.seg[0].bp_plane, bps1 = P.seg[1].bp_plane;
    const bool a_in = va && m0 + BM <= M;
    const bool b_in = (BD || vb) && n0 + BN <= N;
    // KC: thread owns rows x = (tid >> 2) + 64 p (p = 0, 1), k = 4 (tid & 3)
    // .. + 3 (4 lanes per 64-byte row segment).
    // XC: thread owns k pair kp = tid >> 5 (rows 2 kp and 2 kp + 1) and
    // x = 4 (tid & 31) .. + 3 (a wavefront reads 2 whole 512-byte rows).
    const int kx = tid >> 2, ky = 4 * (tid & 3);
    // XC: 4 wavefronts: k pair xk of 4 columns xy..xy+3; 8: of 2 columns
    const int xk = NW == 8 ? tid >> 6 : tid >> 5;
    const int xy = NW == 8 ? 2 * (tid & 63) : 4 * (tid & 31);

    float4 ra[2], rb[2];
    auto load_op = [&](float4 (&r)[2], bool kc, const float* X, int64_t ld,
                       int x0, int X_extent, int k0, int K, bool fast, bool vec) {
      if (kc) {
#pragma unroll
        for (int p = 0; p < AP; ++p) {
          const int x = x0 + kx + 64 * p, k = k0 + ky;
          r[p] = fast ? ld4(X + (int64_t)x * ld + k) : load4(X, ld, x, k, X_extent, K, vec);
        }
      } else if (NW == 8) {  // two columns of rows k, k + 1 in .x, .y
        const int k = k0 + 2 * xk, x = x0 + xy;
        float2 u0, u1;
        if (fast) {
          const float* q = X + (int64_t)k * ld + x;
          u0 = *reinterpret_cast<const float2*>(q);
          u1 = *reinterpret_cast<const float2*>(q + ld);
        } else {
          u0 = load2(X, ld, k, x, K, X_extent, vec);
          u1 = load2(X, ld, k + 1, x, K, X_extent, vec);
        }
        r[0] = make_float4(u0.x, u0.y, 0.f, 0.f);
        r[1] = make_float4(u1.x, u1.y, 0.f, 0.f);
      } else {
        const int k = k0 + 2 * xk, x = x0 + xy;
        if (fast) {
          const float* q = X + (int64_t)k * ld + x;
          r[0] = ld4(q);
          r[1] = ld4(q + ld);
        } else {
          r[0] = load4(X, ld, k, x, K, X_extent, vec);
          r[1] = load4(X, ld, k + 1, x, K, X_extent, vec);
        }
      }
    };
    auto load_slice = [&](int ks) {
      const bool s1 = ks >= kt0;
      const int K = s1 ? K1 : K0;
      const int k0 = (s1 ? ks - kt0 : ks) * BKS;
      const bool fk = k0 + BKS <= K;
      load_op(ra, A_KC, s1 ? A1p : A0p, s1 ? lda1 : lda0, m0, M, k0, K, a_in && fk, va);
      if (!BD)
        load_op(rb, B_KC, s1 ? B1p : B0p, s1 ? ldb1 : ldb0, n0, N, k0, K, b_in && fk, vb);
    };
    // Split this thread's values and write the three pieces.
    auto store_op = [&](uint32_t* L, const float4 (&r)[2], bool kc, int plane) {
      if (kc) {  // 4 consecutive k of rows x and x + 64
#pragma unroll
        for (int p = 0; p < AP; ++p) {
          uint2 h, m, l;
          split3(r[p].x, r[p].y, h.x, m.x, l.x);
          split3(r[p].z, r[p].w, h.y, m.y, l.y);
          const int w = (kx + 64 * p) * KCS_ROW + ky / 2;
          *reinterpret_cast<uint2*>(&L[w]) = h;
          *reinterpret_cast<uint2*>(&L[plane + w]) = m;
          *reinterpret_cast<uint2*>(&L[2 * plane + w]) = l;
        }
      } else if (NW == 8) {  // k pair (rows 2kp, 2kp + 1) of 2 consecutive x
        uint2 h, m, l;
        split3(r[0].x, r[1].x, h.x, m.x, l.x);
        split3(r[0].y, r[1].y, h.y, m.y, l.y);
        const int w = xcs_word(xk, xy);
        *reinterpret_cast<uint2*>(&L[w]) = h;
        *reinterpret_cast<uint2*>(&L[plane + w]) = m;
        *reinterpret_cast<uint2*>(&L[2 * plane + w]) = l;
      } else {   // k pair (rows 2kp, 2kp + 1) of 4 consecutive x
        uint4 h, m, l;
        split3(r[0].x, r[1].x, h.x, m.x, l.x);
        split3(r[0].y, r[1].y, h.y, m.y, l.y);
        split3(r[0].z, r[1].z, h.z, m.z, l.z);
        split3(r[0].w, r[1].w, h.w, m.w, l.w);
        const int w = xcs_word(xk, xy);
        *reinterpret_cast<uint4*>(&L[w]) = h;
        *reinterpret_cast<uint4*>(&L[plane + w]) = m;
        *reinterpret_cast<uint4*>(&L[2 * plane + w]) = l;
      }
    };

    floatx16 acc[2][NJ];
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int j = 0; j < NJ; ++j)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

    // fragment of block i from one piece plane
    auto frag = [&](const uint32_t* L, bool kc, int wbase, int i) {
      uint4 w;
      const int x = wbase + i * 32 + lr;
      if (kc) {
        w = *reinterpret_cast<const uint4*>(&L[x * KCS_ROW + 4 * lh]);
      } else {
        w.x = L[xcs_word(4 * lh + 0, x)];
        w.y = L[xcs_word(4 * lh + 1, x)];
        w.z = L[xcs_word(4 * lh + 2, x)];
        w.w = L[xcs_word(4 * lh + 3, x)];
      }
      return __builtin_bit_cast(bf16x8, w);
    };
    typedef bf16x8 BFr[3][NJ];
    // B fragments of stage ks from the planes (BD); columns past N read as
    // zeros unless `full` (the tile's columns all lie inside N)
    auto load_bfr = [&](BFr& bf, int ks, bool full) {
      const bool s1 = ks >= kt0;
      const uint32_t* Bq = s1 ? Bq1 : Bq0;
      const int64_t ps = s1 ? bps1 : bps0;
      const int64_t gN = (int64_t)(s1 ? ks - kt0 : ks) * N;
#pragma unroll
      for (int j = 0; j < NJ; ++j) {
        const int n = n0 + wn * 32 * NJ + j * 32 + lr;
        const uint32_t* src = Bq + (gN + n) * 8 + 4 * lh;
#pragma unroll
        for (int q = 0; q < 3; ++q) {
          uint4 w = make_uint4(0u, 0u, 0u, 0u);
          if (full || n < N) w = *reinterpret_cast<const uint4*>(src + q * ps);
          bf[q][j] = __builtin_bit_cast(bf16x8, w);
        }
      }
    };
    // The six piece products down to 2^-16 of hi x hi, smallest first; what
    // is left out (mid lo + lo mid + lo lo) is below 2^-24 of |a b|.
    struct Frags {
      bf16x8 a[3][2], b[3][NJ];
    };
    auto read_a = [&](Frags& f, const uint32_t* as) {
#pragma unroll
      for (int q = 0; q < 3; ++q)
#pragma unroll
        for (int i = 0; i < 2; ++i) f.a[q][i] = frag(as + q * A_PLANE, A_KC, wm * 64, i);
    };
    auto read_frags = [&](const uint32_t* as, const uint32_t* bs) {
      Frags f;
      read_a(f, as);
#pragma unroll
      for (int q = 0; q < 3; ++q)
#pragma unroll
        for (int j = 0; j < NJ; ++j) f.b[q][j] = frag(bs + q * B_PLANE, B_KC, wn * 32 * NJ, j);
      return f;
    };
    auto products = [&](const Frags& f) {
      constexpr int terms[6][2] = {{1, 1}, {2, 0}, {0, 2}, {1, 0}, {0, 1}, {0, 0}};
#pragma unroll
      for (int u = 0; u < 6; ++u)
#pragma unroll
        for (int i = 0; i < 2; ++i)
#pragma unroll
          for (int j = 0; j < NJ; ++j)
            acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                f.a[terms[u][0]][i], f.b[terms[u][1]][j], acc[i][j], 0, 0, 0);
    };

    // Stages [kbeg, kf) are full and the tile is interior: pipelined path.
    int kf = kbeg;
    if (a_in && b_in) {
      const int f0 = K0 / BKS, e1 = kt0 + K1 / BKS;
      if (kbeg < f0)
        kf = min(kend, f0 == kt0 ? e1 : f0);
      else if (kbeg >= kt0 && kbeg < e1)
        kf = min(kend, e1);
    }
    if (kf > kbeg) {
      auto load_full = [&](int ks) {
        ks = min(ks, kf - 1);  // past the end: repeat the last stage (never read)
        const bool s1 = ks >= kt0;
        const int k0 = (s1 ? ks - kt0 : ks) * BKS;
        load_op(ra, A_KC, s1 ? A1p : A0p, s1 ? lda1 : lda0, m0, M, k0, 0, true, true);
        if (!BD)
          load_op(rb, B_KC, s1 ? B1p : B0p, s1 ? ldb1 : ldb0, n0, N, k0, 0, true, true);
      };
      if (BD) {
        // A through LDS as below; B fragments of stage k + 1 loaded while
        // stage k's products run (two register sets, alternating)
        BFr b0, b1;
        auto step = [&](const uint32_t* as, uint32_t* as_n, int kl, BFr& bcur,
                        BFr& bnext, int kb) {
          if (second_round)
            __builtin_amdgcn_s_setprio(1);
          else
            __builtin_amdgcn_s_setprio(0);
          Frags f;
          read_a(f, as);
#pragma unroll
          for (int q = 0; q < 3; ++q)
#pragma unroll
            for (int j = 0; j < NJ; ++j) f.b[q][j] = bcur[q][j];
          store_op(as_n, ra, A_KC, A_PLANE);
          load_full(kl);
          load_bfr(bnext, min(kb, kf - 1), true);
          products(f);
          __syncthreads();
        };
        load_full(kbeg);
        store_op(As0, ra, A_KC, A_PLANE);
        load_full(kbeg + 1);
        load_bfr(b0, kbeg, true);
        __syncthreads();
        for (int k = kbeg; k < kf; k += 2) {
          step(As0, As1, k + 2, b0, b1, k + 1);
          if (k + 1 >= kf) break;
          step(As1, As0, k + 3, b1, b0, k + 2);
        }
      } else {
        // Read this stage's fragments, split and store the next stage (in
        // registers) into the other LDS buffer, issue the loads of the stage
        // after it, the products, one barrier.  The fragment reads go first
        // so that the next stage's LDS writes do not hold them up.
        auto step = [&](const uint32_t* as, const uint32_t* bs, uint32_t* as_n,
                        uint32_t* bs_n, int kl) {
          if (second_round && (kl - kbeg) * 10 < (kf - kbeg) * 6)
            __builtin_amdgcn_s_setprio(1);
          else
            __builtin_amdgcn_s_setprio(0);
          const Frags f = read_frags(as, bs);
          store_op(as_n, ra, A_KC, A_PLANE);
          store_op(bs_n, rb, B_KC, B_PLANE);
          load_full(kl);
          products(f);
          __syncthreads();
        };
        load_full(kbeg);
        store_op(As0, ra, A_KC, A_PLANE);
        store_op(Bs0, rb, B_KC, B_PLANE);
        load_full(kbeg + 1);
        __syncthreads();
        for (int k = kbeg; k < kf; k += 2) {
          step(As0, Bs0, As1, Bs1, k + 2);
          if (k + 1 >= kf) break;
          step(As1, Bs1, As0, Bs0, k + 3);
        }
      }
    }

    // Remaining stages (edge tiles, partial K): guarded loads, one stage in
    // registers ahead.
    if (kf < kend) {
      int buf = 0;
      load_slice(kf);
      for (int ks = kf; ks < kend; ++ks) {
        uint32_t* as = buf ? As1 : As0;
        uint32_t* bs = buf ? Bs1 : Bs0;
        store_op(as, ra, A_KC, A_PLANE);
        if (!BD) store_op(bs, rb, B_KC, B_PLANE);
        __syncthreads();
        if (ks + 1 < kend) load_slice(ks + 1);
        if (BD) {
          Frags f;
          read_a(f, as);
          load_bfr(f.b, ks, false);
          products(f);
        } else {
          products(read_frags(as, bs));
        }
        buf ^= 1;
      }
      __syncthreads();
    }

    const bool whole = kbeg == 0 && kend == g.ktiles;
    float* part = g.part + (g.splits > 1 ? (int64_t)lb
                                         : (int64_t)lb * 2 + (seg > 0 ? 1 : 0)) *
                               (BM * BN);
    store_acc<NJ, NW / 2>(P, ti, M, acc, whole, part, wm, wn, lr, lh,
                          g.vec_c[ti.pi] != 0, reinterpret_cast<float*>(As0),
                          reinterpret_cast<float*>(BD || NW == 8 ? As1 : Bs0));
  }
}

// One thread per word (bf16 pair k, k + 1 of one column) of the planes;
// blockIdx.y picks the matrix (job) of the launch.
struct SplitJobs {
  SplitJob j[MAX_SPLIT_JOBS];
  int64_t pw[MAX_SPLIT_JOBS];  // words of one plane of job i
};
__global__ __launch_bounds__(256) void split_b_planes_kernel(SplitJobs jobs) {
  const SplitJob& J = jobs.j[blockIdx.y];
  const int64_t plane_words = jobs.pw[blockIdx.y];
  const int64_t w = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (w >= plane_words) return;
  const float* __restrict__ B = J.B;
  uint32_t* __restrict__ planes = J.planes;
  const int K = J.K, N = J.N;
  const int64_t ld = J.ld;
  const bool kn = !J.trans_b;
  const int tp = (int)(w & 7);
  const int64_t gn = w >> 3;
  const int n = (int)(gn % N), gi = (int)(gn / N);
  const int k = 16 * gi + 2 * tp;
  auto at = [&](int kk) -> float {
    if (kk >= K) return 0.f;
    return kn ? B[(int64_t)kk * ld + n] : B[(int64_t)n * ld + kk];
  };
  uint32_t h, m, l;
  split3(at(k), at(k + 1), h, m, l);
  planes[w] = h;
  planes[plane_words + w] = m;
  planes[2 * plane_words + w] = l;
}

size_t b_planes_words(int32_t K, int32_t N) {
  if (K <= 0 || N <= 0) return 0;
  return 3 * (size_t)ceil_div(K, BKS) * (size_t)N * 8;
}

hipError_t split_b_planes_launch(const SplitJob* jobs, int njobs, hipStream_t s) {
  if (njobs < 1 || njobs > MAX_SPLIT_JOBS) return hipErrorInvalidValue;
  SplitJobs a;
  memset(&a, 0, sizeof(a));
  int64_t pw_max = 0;
  double words = 0;
  for (int i = 0; i < njobs; ++i) {
    a.j[i] = jobs[i];
    const int64_t pw = (int64_t)(b_planes_words(jobs[i].K, jobs[i].N) / 3);
    a.pw[i] = pw;
    pw_max = std::max(pw_max, pw);
    words += (double)pw;
  }
  if (pw_max == 0) return hipSuccess;
  timer_begin(GNN_K_WSPLIT, s);
  split_b_planes_kernel<<<dim3((unsigned)ceil_div(pw_max, 256), (unsigned)njobs), 256, 0, s>>>(a);
  timer_end(GNN_K_WSPLIT, 20.0 * words, s);  // per word: 2 floats in, 3 words out
  return hipGetLastError();
}

// ------------------------------------------------------------------ host

struct Shape {
  int tiles_m, tiles_n0, tiles_n, tiles, ktiles, kt0[2];
  int64_t iters;
  int nblocks;
  int splits;
};

static Shape gemm_shape(const GemmBatch& b) {
  Shape s;
  memset(&s, 0, sizeof(s));
  const int BK = b.mode == GEMM_BF16 ? BK16 : b.mode == GEMM_SPLIT ? BKS : gnnprop::BK;
  const int M = b.p[0].M;
  s.tiles_m = (int)ceil_div(M, BM);
  s.tiles_n0 = (int)ceil_div(b.p[0].N, BN);
  s.tiles_n = s.tiles_n0 + (b.nprob > 1 ? (int)ceil_div(b.p[1].N, BN) : 0);
  s.tiles = s.tiles_m * s.tiles_n;
  for (int i = 0; i < b.nprob; ++i) {
    const GemmProblem& p = b.p[i];
    s.kt0[i] = (int)ceil_div(p.seg[0].K, BK);
    const int kt = s.kt0[i] + (p.nseg > 1 ? (int)ceil_div(p.seg[1].K, BK) : 0);
    s.ktiles = std::max(s.ktiles, kt);
  }
  s.ktiles = std::max(s.ktiles, 1);
  s.iters = (int64_t)s.tiles * s.ktiles;
  // One block per tile when the tiles fill the resident slots well enough.
  // Otherwise, with few tiles and a long K (weight gradients, K = n), split
  // K into S ranges, one (tile, range) per block, ordered split-major so that
  // one XCD's blocks share a K slab of both operands in its L2; with more
  // tiles, split all tile x K-slice iterations evenly over MAX_BLOCKS
  // (the resident slots, 2 per CU).  A launch of few tiles over 4 K slices
  // or more is split even when all its iterations would fit the slots
  // (small weight gradients: 2 tiles over K = 1000 would otherwise walk 32
  // slices one after the other on 2 CUs).  About one tile per CU (224 to
  // 256 tiles) over at most 40 K slices runs one block per tile: measured
  // faster than stream-K plus its reduction (8000 x 512, K = 602: 65.5
  // against 61.3 + 12.2 us), slower from K = 2048 on.  With split products
  // and with bf16 operands the same holds up to one tile per slot over K =
  // 2048 (8000 x 602, K = 1024, 315 tiles: 90.0 us against 89.1 for
  // stream-K with its reduction; bf16 39.2 against 55.1 us), which then
  // writes no partial tiles and needs no second launch; the fp32-MFMA
  // kernel keeps stream-K there (114.0 against 142.4 us).
  // The rules count K in the fp32 kernel's 32-deep slices for the split
  // kernel (two of its 16-deep stages each) and in its own stages for the
  // others (the bf16 kernel's are 64 deep, so its short-K launches stay on
  // one block per tile).
  const int slots = MAX_BLOCKS;
  const int64_t rounds = ceil_div(s.tiles, slots);
  const double fill = (double)s.tiles / (double)(rounds * slots);
  const int kt32 = b.mode == GEMM_SPLIT ? (s.ktiles + 1) / 2 : s.ktiles;
  const int64_t iters32 = (int64_t)s.tiles * kt32;
  const bool one_per_cu = s.tiles >= slots * 7 / 16 &&
                          ((s.tiles <= slots / 2 && kt32 <= 40) ||
                           (b.mode != GEMM_F32 && s.tiles <= slots && kt32 <= 64));
  s.splits = 1;
  if (fill >= 0.85 || one_per_cu ||
      (iters32 <= slots && (s.tiles > slots / 4 || kt32 < 4))) {
    s.nblocks = s.tiles;
  } else if (s.tiles <= slots / 4) {
    s.splits = (int)std::min<int64_t>(s.ktiles, slots / s.tiles);
    s.nblocks = s.tiles * s.splits;
  } else {
    // stream-K: every block gets at least one K slice, so that the blocks
    // sharing a tile are consecutive and each holds a partial of it
    s.nblocks = (int)std::min<int64_t>(slots, s.iters);
  }
  return s;
}

static bool batch_ok(const GemmBatch& b) {
  if (b.nprob < 1 || b.nprob > 2) return false;
  const int BK = b.mode == GEMM_BF16 ? BK16 : b.mode == GEMM_SPLIT ? BKS : gnnprop::BK;
  if (b.nprob == 2) {
    if (b.p[0].M != b.p[1].M) return false;
    const auto kt = [BK](const GemmProblem& p) {
      return ceil_div(p.seg[0].K, BK) + (p.nseg > 1 ? ceil_div(p.seg[1].K, BK) : 0);
    };
    if (kt(b.p[0]) != kt(b.p[1])) return false;
  }
  return true;
}

size_t gemm_workspace_bytes(const GemmBatch& b) {
  if (!batch_ok(b)) return 0;
  const Shape s = gemm_shape(b);
  if (s.tiles == 0 || s.nblocks == s.tiles) return 0;
  const size_t slots = s.splits > 1 ? (size_t)s.nblocks : (size_t)s.nblocks * 2;
  return round_up(slots * BM * BN * 4, 256);
}

double gemm_flops(const GemmBatch& b) {
  double f = 0;
  for (int i = 0; i < b.nprob; ++i) {
    const GemmProblem& p = b.p[i];
    for (int s = 0; s < p.nseg; ++s) f += 2.0 * p.M * p.N * (double)p.seg[s].K;
  }
  return f;
}

// The reduction of a launch's shared tiles as its own kernel.
static hipError_t fixup_launch(const GemmKArgs& g, hipStream_t s) {
  timer_begin(GNN_K_GEMM_REDUCE, s);
  gemm_fixup_kernel<<<dim3((unsigned)g.tiles, FIX_CHUNKS), 256, 0, s>>>(g);
  timer_end(GNN_K_GEMM_REDUCE, 0.0, s);
  return hipGetLastError();
}

hipError_t gemm_flush(const GemmFixup& fx, hipStream_t s) {
  if (!fx.pending) return hipSuccess;
  GemmKArgs g;
  memcpy(&g, fx.args, sizeof(g));
  return fixup_launch(g, s);
}

hipError_t gemm_launch(const GemmBatch& b, void* workspace, size_t ws_bytes,
                       hipStream_t s, GemmFixup* defer, const GemmFixup* pending) {
  static_assert(sizeof(GemmKArgs) <= sizeof(GemmFixup::args), "GemmFixup size");
  if (defer) defer->pending = 0;
  if (!batch_ok(b)) return hipErrorInvalidValue;
  // bf16-stored operands: the bf16 mode's weight-gradient (B) and
  // input-gradient (A) launches only
  if (b.a16 || b.b16) {
    if (b.mode != GEMM_BF16 || (b.a16 && b.b16)) return hipErrorInvalidValue;
    if (b.b16 && !(b.trans_a && !b.trans_b)) return hipErrorInvalidValue;
    if (b.a16 && !(!b.trans_a && b.trans_b)) return hipErrorInvalidValue;
  }
  if (b.b_planes) {  // split products only, every segment's planes given
    if (b.mode != GEMM_SPLIT) return hipErrorInvalidValue;
    for (int i = 0; i < b.nprob; ++i)
      for (int k = 0; k < b.p[i].nseg; ++k)
        if (b.p[i].seg[k].K > 0 && !b.p[i].seg[k].Bp) return hipErrorInvalidValue;
  }
  const Shape sh = gemm_shape(b);
  if (sh.tiles == 0) return pending ? gemm_flush(*pending, s) : hipSuccess;
  GemmKArgs g;
  memset(&g, 0, sizeof(g));
  g.nprob = b.nprob;
  g.M = b.p[0].M;
  g.tiles_m = sh.tiles_m;
  g.tiles_n0 = sh.tiles_n0;
  g.tiles_n = sh.tiles_n;
  g.tiles = sh.tiles;
  g.ktiles = sh.ktiles;
  g.iters = sh.iters;
  g.nblocks = sh.nblocks;
  g.splits = sh.splits;
  bool va = true, vb = true;
  // 4 consecutive elements per load: 16 bytes (fp32) or 8 (bf16 storage)
  auto vec_ok = [](const void* p, int64_t ld, bool h) {
    return h ? (reinterpret_cast<uintptr_t>(p) % 8 == 0 && ld % 4 == 0) : vec4_ok(p, ld);
  };
  for (int i = 0; i < b.nprob; ++i) {
    g.p[i] = b.p[i];
    if (g.p[i].nseg < 2) {
      g.p[i].seg[1] = g.p[i].seg[0];
      g.p[i].seg[1].K = 0;
    }
    g.ktiles0[i] = sh.kt0[i];
    const GemmProblem& p = g.p[i];
    for (int k = 0; k < p.nseg; ++k) {
      va = va && vec_ok(p.seg[k].A, p.seg[k].lda, b.a16 != 0);
      vb = vb && vec_ok(p.seg[k].B, p.seg[k].ldb, b.b16 != 0);
    }
  }
  for (int i = 0; i < b.nprob; ++i) {
    const GemmProblem& p = g.p[i];
    g.vec_c[i] = vec4_ok(p.C, p.ldc) && (!p.mask || vec4_ok(p.mask, p.ld_mask)) &&
                 (!p.bias || aligned16(p.bias));
  }
  g.vec_a = va;
  g.vec_b = vb;
  const bool streamk = sh.nblocks != sh.tiles;
  if (streamk) {
    if (ws_bytes < gemm_workspace_bytes(b) || !workspace)
      return hipErrorInvalidValue;
    g.part = static_cast<float*>(workspace);
  }
  // a reduction left by the previous launch: its chunks as extra blocks
  GemmKArgs fx;
  memset(&fx, 0, sizeof(fx));
  int extra = 0;
  if (pending && pending->pending) {
    memcpy(&fx, pending->args, sizeof(fx));
    extra = fx.tiles * FIX_CHUNKS;
  }
  const unsigned grid = (unsigned)(sh.nblocks + extra);
  const int kid = b.trans_a ? (b.trans_b ? GNN_K_GEMM_TT : GNN_K_GEMM_TN)
                            : (b.trans_b ? GNN_K_GEMM_NT : GNN_K_GEMM_NN);
  timer_begin(kid, s);
  if (b.mode == GEMM_BF16 && b.b16) {  // (checked above: trans_a, !trans_b, !a16)
    gemm_bf16_kernel<true, false, false, true><<<grid, 256, 0, s>>>(g, fx);
  } else if (b.mode == GEMM_BF16 && b.a16) {  // (!trans_a, trans_b)
    gemm_bf16_kernel<false, true, true, false><<<grid, 256, 0, s>>>(g, fx);
  } else if (b.mode == GEMM_BF16) {
    if (!b.trans_a && !b.trans_b)
      gemm_bf16_kernel<false, false, false, false><<<grid, 256, 0, s>>>(g, fx);
    else if (b.trans_a && !b.trans_b)
      gemm_bf16_kernel<true, false, false, false><<<grid, 256, 0, s>>>(g, fx);
    else if (!b.trans_a && b.trans_b)
      gemm_bf16_kernel<false, true, false, false><<<grid, 256, 0, s>>>(g, fx);
    else
      gemm_bf16_kernel<true, true, false, false><<<grid, 256, 0, s>>>(g, fx);
  } else if (b.mode == GEMM_F32) {
    if (!b.trans_a && !b.trans_b)
      gemm_f32_kernel<false, false><<<grid, 256, 0, s>>>(g, fx);
    else if (b.trans_a && !b.trans_b)
      gemm_f32_kernel<true, false><<<grid, 256, 0, s>>>(g, fx);
    else if (!b.trans_a && b.trans_b)
      gemm_f32_kernel<false, true><<<grid, 256, 0, s>>>(g, fx);
    else
      gemm_f32_kernel<true, true><<<grid, 256, 0, s>>>(g, fx);
  } else if (b.b_planes && !b.trans_a) {
    if (!b.trans_b)
      gemm_split_kernel<false, false, true, 8><<<grid, 512, 0, s>>>(g, fx);
    else
      gemm_split_kernel<false, true, true, 8><<<grid, 512, 0, s>>>(g, fx);
  } else if (b.b_planes) {
    if (!b.trans_a && !b.trans_b)
      gemm_split_kernel<false, false, true><<<grid, 256, 0, s>>>(g, fx);
    else if (b.trans_a && !b.trans_b)
      gemm_split_kernel<true, false, true><<<grid, 256, 0, s>>>(g, fx);
    else if (!b.trans_a && b.trans_b)
      gemm_split_kernel<false, true, true><<<grid, 256, 0, s>>>(g, fx);
    else
      gemm_split_kernel<true, true, true><<<grid, 256, 0, s>>>(g, fx);
  } else if (!b.trans_a && !b.trans_b) {
    gemm_split_kernel<false, false, false, 8><<<grid, 512, 0, s>>>(g, fx);
  } else if (b.trans_a && !b.trans_b) {
    gemm_split_kernel<true, false, false><<<grid, 256, 0, s>>>(g, fx);
  } else if (!b.trans_a && b.trans_b) {
    gemm_split_kernel<false, true, false, 8><<<grid, 512, 0, s>>>(g, fx);
  } else {
    gemm_split_kernel<true, true, false><<<grid, 256, 0, s>>>(g, fx);
  }
  timer_end(kid, gemm_flops(b), s);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || !streamk) return e;
  if (defer) {  // the next launch (or gemm_flush) sums the shared tiles
    memcpy(defer->args, &g, sizeof(g));
    defer->pending = 1;
    return hipSuccess;
  }
  return fixup_launch(g, s);
}

}  // namespace gnnprop
