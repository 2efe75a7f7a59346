// Internal interfaces between the translation units of libgnnprop.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <algorithm>
#include <cstring>

#include "gnnprop.h"

namespace gnnprop {

// --------------------------------------------------------------- helpers

__host__ __device__ inline int64_t ceil_div(int64_t a, int64_t b) {
  return (a + b - 1) / b;
}
__host__ __device__ inline int64_t round_up(int64_t a, int64_t b) {
  return ceil_div(a, b) * b;
}
inline bool aligned16(const void* p) {
  return (reinterpret_cast<uintptr_t>(p) & 15u) == 0;
}
// Row-major matrix that may be read/written with float4 accesses.
inline bool vec4_ok(const void* p, int64_t ld) {
  return p != nullptr && aligned16(p) && (ld % 4) == 0;
}

// ------------------------------------------------------------ work plan

// Layout of the aggregation plan buffer (device memory), at the offsets of
// plan_dims():
//   PlanHeader;
//   int4 binfo[nblk]  per aggregation workgroup: rows [x, y) and their
//                     entries [z, w); the rows whose first entry lies in
//                     window [k, k+1) * block_entries;
//   int32 erow[nnz]   row of each entry.
struct PlanHeader {
  int32_t nblk;
  int32_t block_entries;
  int32_t n;
  int32_t nnz;
  int32_t pad[4];
};

struct PlanDims {
  int32_t block_entries;
  int64_t nblk;
  size_t binfo_offset, erow_offset, bytes;
};
PlanDims plan_dims(int32_t n, int64_t nnz);

// ------------------------------------------------------- kernel timing

struct Timer;
// Records `start`/`stop` events around the launch when timing is enabled.
void timer_begin(int kclass, hipStream_t s);
void timer_end(int kclass, double work, hipStream_t s);

// ------------------------------------------------------------ SpMM

enum SpmmEpilogue : int32_t {
  SPMM_STORE = 0,      // out = acc
  SPMM_BIAS_RELU = 1,  // out = max(acc + bias[c], 0)   (bias may be null)
  SPMM_ADD = 2,        // out = acc + res[row, c]         (res may alias out)
  SPMM_STORE_BF16 = 3, // out = acc rounded to bf16 (uint16 storage; rows
                       // 8-byte aligned, ld_out a multiple of 4 elements)
};                     // with `mask` set: out = mask[row, c] > 0 ? out : 0

// Where the weight of a stored entry comes from:
//   SPMM_W_VALUES    the value array (vals);
//   SPMM_W_ROW_SCALE A = D^-1 B with B the 0/1 pattern: the entries of a row
//                    are summed unweighted and the sum is scaled by 1/deg of
//                    that row (deg = its stored entries) when the row is
//                    written; vals is not read;
//   SPMM_W_COL_DEG   (D^-1 B)^T on a symmetric pattern: entry (u, v) weighs
//                    1/deg(v), taken from the row pointers; vals is not read.
enum SpmmWeights : int32_t { SPMM_W_VALUES = 0, SPMM_W_ROW_SCALE = 1, SPMM_W_COL_DEG = 2 };

struct SpmmCall {
  int32_t n;
  int64_t nnz;
  const int32_t* indptr;
  const int32_t* indices;
  const float* vals;
  const void* plan;
  int32_t w;
  const float* in;
  int64_t ld_in;
  float* out;
  int64_t ld_out;
  int32_t epilogue;
  const float* bias;
  const float* res;
  int64_t ld_res;
  const float* mask;
  int64_t ld_mask;
  int32_t weights;  // SpmmWeights
};
size_t spmm_partials_bytes(int32_t n, int64_t nnz, int32_t w);
hipError_t spmm_launch(const SpmmCall& c, hipStream_t s);
// The aggregation's loads and gathers alone (a measurement floor; float4
// lanes only: hipErrorInvalidValue when rows are not 16-byte aligned).
hipError_t spmm_floor_launch(const SpmmCall& c, hipStream_t s);

hipError_t plan_build_launch(int32_t n, int64_t nnz, const int32_t* indptr,
                             const int32_t* indices, void* plan, hipStream_t s);
// One thread per entry (rows from the plan) when `plan` is non-null (built
// for this graph), else one wavefront per row.
hipError_t transpose_values_launch(int32_t n, int64_t nnz,
                                   const int32_t* indptr,
                                   const int32_t* indices, const float* vals,
                                   float* vals_t, const void* plan,
                                   hipStream_t s);
// Plan and transposed values of one graph in a single launch.
hipError_t prepare_launch(int32_t n, int64_t nnz, const int32_t* indptr,
                          const int32_t* indices, const float* vals,
                          float* vals_t, void* plan, hipStream_t s);
// Returns 0 if valid, else a nonzero code; synchronises.
hipError_t validate_csr(int32_t n, int64_t nnz, const int32_t* indptr,
                        const int32_t* indices, int32_t symmetric,
                        int32_t* bad, hipStream_t s);

// ------------------------------------------------------------ GEMM

// C = sum over segments of op(A_s) op(B_s), then + bias[col], then ReLU.
struct GemmSeg {
  const float* A;
  const float* B;
  int64_t lda, ldb;
  int32_t K;
  // Split mode with GemmBatch::b_planes: op(B) already split into its three
  // bf16 pieces in fragment order (split_b_planes_launch); B is not read.
  const uint32_t* Bp = nullptr;
  int64_t bp_plane = 0;  // 32-bit words between two pieces' planes
};
struct GemmProblem {
  GemmSeg seg[2];
  int32_t nseg;
  int32_t M, N;
  float* C;
  int64_t ldc;
  const float* bias;
  int32_t relu;
  const float* mask;  // if set: C = mask[r, c] > 0 ? C : 0 (after bias/ReLU)
  int64_t ld_mask;
};
// How the products are formed (fp32 accumulation in every mode):
//   GEMM_SPLIT  fp32 operands as three bf16 pieces each, six piece products
//               on the bf16 matrix cores (the default; fp32 accuracy);
//   GEMM_BF16   operands rounded to bf16, one product (GNN_FLAG_BF16);
//   GEMM_F32    the fp32 matrix-core instruction (GNN_FLAG_F32_MFMA).
enum GemmMode : int32_t { GEMM_SPLIT = 0, GEMM_BF16 = 1, GEMM_F32 = 2 };
constexpr uint32_t GEMM_FLAGS = GNN_FLAG_BF16 | GNN_FLAG_F32_MFMA;
inline int32_t gemm_mode(uint32_t flags) {
  return (flags & GNN_FLAG_BF16) ? GEMM_BF16
                                 : (flags & GNN_FLAG_F32_MFMA) ? GEMM_F32 : GEMM_SPLIT;
}
// Both product flags at once is not a mode.
inline bool gemm_flags_ok(uint32_t flags) {
  return (flags & GEMM_FLAGS) != GEMM_FLAGS;
}
struct GemmBatch {
  GemmProblem p[2];
  int32_t nprob;
  int32_t trans_a, trans_b;  // A stored K x M; B stored N x K
  int32_t mode;              // GemmMode
  int32_t b_planes;          // split mode: every segment's B given as Bp
  // bf16 mode: every segment's A (a16) or B (b16) holds bf16 values (the
  // float pointer points at them, ld in elements); supported for the weight
  // gradients' B (trans_a, !trans_b) and the input gradient's A (trans_b)
  int32_t a16, b16;
};
// op(B) (K x N; stored K x N row-major when !trans_b, N x K when trans_b,
// row stride ld) split exactly into bf16 hi + mid + lo (each rounded to
// nearest even), written as three planes in MFMA fragment order: plane q,
// 16-deep group g = k / 16, column n: the 16 pieces of k = 16 g .. 16 g + 15
// as 8 words of bf16 pairs, at words ((g N + n) 8 .. + 7) of the plane; k
// past K holds zeros.  Planes are b_planes_words(K, N) / 3 words apart.
size_t b_planes_words(int32_t K, int32_t N);
// One matrix to split: op(B) (K x N) of B with row stride ld, into the
// planes at `planes` (b_planes_words(K, N) words, 16-byte aligned).
struct SplitJob {
  const float* B;
  int64_t ld;
  int32_t K, N;
  int32_t trans_b;
  uint32_t* planes;
};
constexpr int MAX_SPLIT_JOBS = 4;
// Up to MAX_SPLIT_JOBS matrices split in one launch.
hipError_t split_b_planes_launch(const SplitJob* jobs, int njobs, hipStream_t s);
size_t gemm_workspace_bytes(const GemmBatch& b);
// The reduction of a stream-K or split-K launch's shared tiles, held back so
// that the next GEMM launch on the stream runs it in extra blocks of its own
// grid instead of a kernel of its own.  The held launch's partial tiles
// (its workspace) must stay untouched until then: the next launch takes
// another workspace region.
struct GemmFixup {
  int32_t pending = 0;
  alignas(16) unsigned char args[512];  // the held launch's kernel arguments
};
// `defer`: if the launch needs a reduction, hold it in *defer instead of
// running it.  `pending`: a held reduction to run in this launch (or alone
// when this launch has no tiles).
hipError_t gemm_launch(const GemmBatch& b, void* workspace, size_t ws_bytes,
                       hipStream_t s, GemmFixup* defer = nullptr,
                       const GemmFixup* pending = nullptr);
// Runs a held reduction as a kernel of its own (no-op if none is held).
hipError_t gemm_flush(const GemmFixup& fx, hipStream_t s);
double gemm_flops(const GemmBatch& b);

// ----------------------------------------------------- elementwise

typedef __bf16 bf16x2v __attribute__((ext_vector_type(2)));
// Two floats rounded to bf16 (round to nearest even), packed low, high.
__device__ inline uint32_t pack_bf16(float lo, float hi) {
  bf16x2v v = {(__bf16)lo, (__bf16)hi};
  return __builtin_bit_cast(uint32_t, v);
}

// G = dY * 1[Y > 0] over an n x width block; columns [0, split) -> dst0,
// [split, width) -> dst1 (dst1 unused when split = width).  dst0_bf16:
// dst0 receives G rounded to bf16 (uint16 storage, ld0 in elements).
hipError_t mask_launch(int32_t n, int32_t width, int32_t split,
                       const float* Y, const float* dY, int64_t ld_y,
                       void* dst0, int64_t ld0, float* dst1, int64_t ld1,
                       hipStream_t s, bool dst0_bf16 = false);
// out[c] = sum over rows of G[r, c] in a fixed order (the same for every
// call with the same n); with row_weight, out[c] = sum_r row_weight[r] G[r, c].
// colsum2 forms out0 = G^T w0 and out1 = G^T w1 from one pass over G.
// partials: colsum_partials_bytes(n, w, number of sums).
size_t colsum_partials_bytes(int32_t n, int32_t w, int nw = 1);
hipError_t colsum_launch(int32_t n, int32_t w, const float* G, int64_t ldg,
                         float* out, float* partials, hipStream_t s,
                         const float* row_weight = nullptr);
hipError_t colsum2_launch(int32_t n, int32_t w, const float* G, int64_t ldg,
                          const float* w0, const float* w1, float* out0,
                          float* out1, float* partials, hipStream_t s);
// out[c] = sum over rows of (Y[r, c] > 0 ? dY[r, c] : 0), the bias gradient
// taken from the layer's output and its gradient directly (same order as
// colsum_launch of the masked G).
hipError_t colsum_masked_launch(int32_t n, int32_t w, const float* Y, const float* dY,
                                int64_t ld, float* out, float* partials, hipStream_t s);

}  // namespace gnnprop
