// Sparse feature / gradient propagation on gfx950 (the first of the three
// kernels of Section 5.1) and the per-subgraph preparation it needs: the
// degree-binned work plan and the transposed value array of Section 5.2
// (Algorithm 6).
//
// Aggregation design.  Row v of A_s . X is the weighted sum of the input
// rows of v's neighbours.  One wavefront-group of G lanes owns one work item
// (a whole row, or a chunk of at most `chunk` stored entries of a long row)
// and sweeps the feature columns with float4 loads, so every gathered
// neighbour row is read as whole 64-byte segments.  Power-law subgraphs
// have a few rows with thousands of entries; the plan cuts those into
// chunks processed by separate wavefronts, whose partial rows a second
// kernel adds in chunk order (no atomics, bit-reproducible).  The paper's
// column partition (Algorithm 7) is what each group's column sweep does
// within a row; its cache-size rule is left to the L2/MALL hierarchy.
#include "internal.hpp"

namespace gnnprop {

// ------------------------------------------------------------ plan sizes

static int32_t plan_chunk(int32_t n, int64_t nnz) {
  (void)n;
  (void)nnz;
  return 64;
}

PlanDims plan_dims(int32_t n, int64_t nnz) {
  PlanDims d;
  d.chunk = plan_chunk(n, nnz);
  const int64_t q = ceil_div(nnz, d.chunk);
  d.max_items = (int64_t)n + q;        // sum of max(1, ceil(deg/chunk))
  d.max_splits = nnz / (d.chunk + 1);  // rows with deg > chunk
  // sum of ceil(deg/chunk) over the split rows
  d.max_slots = d.max_splits > 0 ? q + d.max_splits : 0;
  d.items_offset = round_up(sizeof(PlanHeader), 256);
  d.splits_offset = round_up(d.items_offset + 16 * (size_t)d.max_items, 256);
  d.tot_offset = round_up(d.splits_offset + 16 * (size_t)(d.max_splits + 1), 256);
  d.bytes = round_up(d.tot_offset + 12 * (size_t)(ceil_div(n, 2048) + 1), 256);
  return d;
}

// ----------------------------------------------------------- plan build
//
// Two passes over the row pointers, 2048 rows per block: the first counts
// each block's items, split rows and partial slots; the second turns those
// block totals into prefixes, scans within the block and writes the items.

constexpr int PB_THREADS = 256;
constexpr int PB_ROWS = 8;
constexpr int PB_BLOCK_ROWS = PB_THREADS * PB_ROWS;

struct RowCounts {
  int c[3];  // items, split rows, partial slots
};

__device__ inline RowCounts count_rows(const int32_t* __restrict__ indptr,
                                       int32_t n, int32_t chunk, int64_t r0) {
  RowCounts rc = {{0, 0, 0}};
  for (int k = 0; k < PB_ROWS; ++k) {
    const int64_t r = r0 + k;
    if (r < n) {
      const int d = indptr[r + 1] - indptr[r];
      if (d > chunk) {
        const int nch = (d + chunk - 1) / chunk;
        rc.c[0] += nch;
        rc.c[1] += 1;
        rc.c[2] += nch;
      } else {
        rc.c[0] += 1;
      }
    }
  }
  return rc;
}

__device__ inline int wave_incl_scan(int x) {
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int d = 1; d < 64; d <<= 1) {
    const int y = __shfl_up(x, d, 64);
    if (lane >= d) x += y;
  }
  return x;
}

// Exclusive prefix sums of three counters over the block, plus totals.
__device__ inline void block_scan3(const int v[3], int excl[3], int tot[3],
                                   int (*s_w)[3]) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  constexpr int NW = PB_THREADS / 64;
  int inc[3];
#pragma unroll
  for (int k = 0; k < 3; ++k) inc[k] = wave_incl_scan(v[k]);
  if (lane == 63)
    for (int k = 0; k < 3; ++k) s_w[wave][k] = inc[k];
  __syncthreads();
  if (threadIdx.x < 3) {
    int run = 0;
    for (int w = 0; w < NW; ++w) {
      const int x = s_w[w][threadIdx.x];
      s_w[w][threadIdx.x] = run;
      run += x;
    }
    s_w[NW][threadIdx.x] = run;
  }
  __syncthreads();
#pragma unroll
  for (int k = 0; k < 3; ++k) {
    excl[k] = s_w[wave][k] + inc[k] - v[k];
    tot[k] = s_w[NW][k];
  }
}

__global__ __launch_bounds__(PB_THREADS) void plan_count_kernel(
    const int32_t* __restrict__ indptr, int32_t n, int32_t chunk,
    int32_t* __restrict__ block_tot) {
  __shared__ int s_w[PB_THREADS / 64 + 1][3];
  const int64_t r0 = (int64_t)blockIdx.x * PB_BLOCK_ROWS + threadIdx.x * PB_ROWS;
  const RowCounts rc = count_rows(indptr, n, chunk, r0);
  int excl[3], tot[3];
  block_scan3(rc.c, excl, tot, s_w);
  if (threadIdx.x == 0)
    for (int k = 0; k < 3; ++k) block_tot[blockIdx.x * 3 + k] = tot[k];
}

__global__ __launch_bounds__(PB_THREADS) void plan_fill_kernel(
    const int32_t* __restrict__ indptr, int32_t n, int32_t chunk,
    const int32_t* __restrict__ block_tot, int4* __restrict__ items,
    int4* __restrict__ splits, PlanHeader* __restrict__ hdr) {
  __shared__ int s_w[PB_THREADS / 64 + 1][3];
  __shared__ int s_pre[3];
  if (threadIdx.x < 3) {  // prefix over the earlier blocks, in block order
    int run = 0;
    for (int b = 0; b < (int)blockIdx.x; ++b) run += block_tot[b * 3 + threadIdx.x];
    s_pre[threadIdx.x] = run;
  }
  const int64_t r0 = (int64_t)blockIdx.x * PB_BLOCK_ROWS + threadIdx.x * PB_ROWS;
  const RowCounts rc = count_rows(indptr, n, chunk, r0);
  int excl[3], tot[3];
  block_scan3(rc.c, excl, tot, s_w);  // its barriers also publish s_pre
  int oi = s_pre[0] + excl[0], os = s_pre[1] + excl[1], ol = s_pre[2] + excl[2];
  for (int k = 0; k < PB_ROWS; ++k) {
    const int64_t r = r0 + k;
    if (r < n) {
      const int b = indptr[r], e = indptr[r + 1], d = e - b;
      if (d > chunk) {
        const int nch = (d + chunk - 1) / chunk;
        splits[os++] = make_int4((int)r, ol, nch, 0);
        for (int c = 0; c < nch; ++c) {
          const int cb = b + c * chunk;
          items[oi++] = make_int4((int)r, cb, min(e, cb + chunk), ol + c);
        }
        ol += nch;
      } else {
        items[oi++] = make_int4((int)r, b, e, -1);
      }
    }
  }
  if (blockIdx.x == gridDim.x - 1 && threadIdx.x == 0) {
    PlanHeader h;
    h.n_items = s_pre[0] + tot[0];
    h.n_splits = s_pre[1] + tot[1];
    h.chunk = chunk;
    h.n_slots = s_pre[2] + tot[2];
    h.n = n;
    h.pad[0] = h.pad[1] = h.pad[2] = 0;
    *hdr = h;
  }
}

hipError_t plan_build_launch(int32_t n, int64_t nnz, const int32_t* indptr,
                             void* plan, hipStream_t s) {
  const PlanDims d = plan_dims(n, nnz);
  char* base = static_cast<char*>(plan);
  const unsigned nb = (unsigned)std::max<int64_t>(1, ceil_div(n, PB_BLOCK_ROWS));
  int32_t* tot = reinterpret_cast<int32_t*>(base + d.tot_offset);
  timer_begin(GNN_K_PLAN, s);
  plan_count_kernel<<<nb, PB_THREADS, 0, s>>>(indptr, n, d.chunk, tot);
  plan_fill_kernel<<<nb, PB_THREADS, 0, s>>>(
      indptr, n, d.chunk, tot, reinterpret_cast<int4*>(base + d.items_offset),
      reinterpret_cast<int4*>(base + d.splits_offset),
      reinterpret_cast<PlanHeader*>(base));
  timer_end(GNN_K_PLAN, 8.0 * (n + 1) + 16.0 * n, s);
  return hipGetLastError();
}

// ---------------------------------------------- transposed values (Alg. 6)

// Stored entry (v,u) of A_s is entry (u,v) of the transpose, which lives in
// row u at the position of column v.  Rows are sorted, so that position is
// found by binary search; every entry is moved exactly once.
__device__ inline void transpose_entry(int v, int j, const int32_t* indptr,
                                       const int32_t* indices,
                                       const float* vals, float* vals_t) {
  const int u = indices[j];
  int lo = indptr[u], hi = indptr[u + 1];
  const int end = hi;
  while (lo < hi) {
    const int mid = (lo + hi) >> 1;
    if (indices[mid] < v)
      lo = mid + 1;
    else
      hi = mid;
  }
  if (lo < end && indices[lo] == v) vals_t[lo] = vals[j];
}

// One wavefront per row.
__global__ __launch_bounds__(256) void transpose_values_kernel(
    int32_t n, const int32_t* __restrict__ indptr,
    const int32_t* __restrict__ indices, const float* __restrict__ vals,
    float* __restrict__ vals_t) {
  const int v = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (v >= n) return;
  const int lane = threadIdx.x & 63;
  const int b = indptr[v], e = indptr[v + 1];
  for (int j = b + lane; j < e; j += 64)
    transpose_entry(v, j, indptr, indices, vals, vals_t);
}

// One wavefront per work item of the aggregation plan (at most `chunk`
// entries), so a hub row is spread over many wavefronts.
__global__ __launch_bounds__(256) void transpose_values_items_kernel(
    const PlanHeader* __restrict__ hdr, const int4* __restrict__ items,
    const int32_t* __restrict__ indptr, const int32_t* __restrict__ indices,
    const float* __restrict__ vals, float* __restrict__ vals_t) {
  const int i = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (i >= hdr->n_items) return;
  const int4 it = items[i];
  const int lane = threadIdx.x & 63;
  for (int j = it.y + lane; j < it.z; j += 64)
    transpose_entry(it.x, j, indptr, indices, vals, vals_t);
}

hipError_t transpose_values_launch(int32_t n, int64_t nnz,
                                   const int32_t* indptr,
                                   const int32_t* indices, const float* vals,
                                   float* vals_t, const void* plan,
                                   hipStream_t s) {
  if (n <= 0) return hipSuccess;
  timer_begin(GNN_K_TRANSPOSE, s);
  if (plan) {
    const PlanDims d = plan_dims(n, nnz);
    const char* base = static_cast<const char*>(plan);
    transpose_values_items_kernel<<<(unsigned)ceil_div(d.max_items, 4), 256, 0, s>>>(
        reinterpret_cast<const PlanHeader*>(base),
        reinterpret_cast<const int4*>(base + d.items_offset), indptr, indices,
        vals, vals_t);
  } else {
    transpose_values_kernel<<<(unsigned)ceil_div(n, 4), 256, 0, s>>>(
        n, indptr, indices, vals, vals_t);
  }
  timer_end(GNN_K_TRANSPOSE, 0.0, s);
  return hipGetLastError();
}

// --------------------------------------------------------------- validate

__global__ __launch_bounds__(256) void validate_kernel(
    int32_t n, int64_t nnz, const int32_t* __restrict__ indptr,
    const int32_t* __restrict__ indices, int32_t symmetric,
    int32_t* __restrict__ bad) {
  const int64_t r = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (r == 0 && (indptr[0] != 0 || (int64_t)indptr[n] != nnz)) bad[0] = 1;
  if (r >= n) return;
  const int64_t b = indptr[r], e = indptr[r + 1];
  if (b < 0 || e > nnz || e < b) {
    bad[0] = 2;
    return;
  }
  int prev = -1;
  for (int64_t j = b; j < e; ++j) {
    const int u = indices[j];
    if (u < 0 || u >= n || u <= prev) {
      bad[0] = 3;
      return;
    }
    prev = u;
    if (symmetric) {
      int64_t lo = indptr[u], hi = indptr[u + 1];
      if (lo < 0 || hi > nnz || hi < lo) {
        bad[0] = 2;
        return;
      }
      const int64_t end = hi;
      while (lo < hi) {
        const int64_t mid = (lo + hi) >> 1;
        if (indices[mid] < (int)r)
          lo = mid + 1;
        else
          hi = mid;
      }
      if (!(lo < end && indices[lo] == (int)r)) {
        bad[0] = 4;
        return;
      }
    }
  }
}

hipError_t validate_csr(int32_t n, int64_t nnz, const int32_t* indptr,
                        const int32_t* indices, int32_t symmetric,
                        int32_t* bad, hipStream_t s) {
  const unsigned grid = (unsigned)(n > 0 ? ceil_div(n, 256) : 1);
  validate_kernel<<<grid, 256, 0, s>>>(n, nnz, indptr, indices, symmetric,
                                        bad);
  return hipGetLastError();
}

// ------------------------------------------------------------- aggregation

struct SpmmArgs {
  const int32_t* indices;
  const float* vals;
  const PlanHeader* hdr;
  const int4* items;
  const int4* splits;
  int32_t w;
  const float* in;
  int64_t ld_in;
  float* out;
  int64_t ld_out;
  int32_t epilogue;
  const float* bias;
  const float* res;
  int64_t ld_res;
  float* part;
  int64_t ldp;
  int32_t nslices;  // column slices (blocks b with b % nslices == q own slice q)
  int32_t sw;       // slice width in columns
};

template <bool VEC>
struct Vec;
template <>
struct Vec<true> {
  using T = float4;
  static constexpr int W = 4;
  __device__ static T zero() { return make_float4(0.f, 0.f, 0.f, 0.f); }
  __device__ static T load(const float* p) {
    return *reinterpret_cast<const float4*>(p);
  }
  __device__ static void store(float* p, T v) {
    *reinterpret_cast<float4*>(p) = v;
  }
  __device__ static void fma(T& acc, float a, T x) {
    acc.x = fmaf(a, x.x, acc.x);
    acc.y = fmaf(a, x.y, acc.y);
    acc.z = fmaf(a, x.z, acc.z);
    acc.w = fmaf(a, x.w, acc.w);
  }
  __device__ static void add(T& acc, T x) {
    acc.x += x.x;
    acc.y += x.y;
    acc.z += x.z;
    acc.w += x.w;
  }
  __device__ static T bias_relu(T v, const float* b) {
    if (b) {
      const float4 bb = *reinterpret_cast<const float4*>(b);
      v.x += bb.x;
      v.y += bb.y;
      v.z += bb.z;
      v.w += bb.w;
    }
    v.x = fmaxf(v.x, 0.f);
    v.y = fmaxf(v.y, 0.f);
    v.z = fmaxf(v.z, 0.f);
    v.w = fmaxf(v.w, 0.f);
    return v;
  }
};
template <>
struct Vec<false> {
  using T = float;
  static constexpr int W = 1;
  __device__ static T zero() { return 0.f; }
  __device__ static T load(const float* p) { return *p; }
  __device__ static void store(float* p, T v) { *p = v; }
  __device__ static void fma(T& acc, float a, T x) { acc = fmaf(a, x, acc); }
  __device__ static void add(T& acc, T x) { acc += x; }
  __device__ static T bias_relu(T v, const float* b) {
    if (b) v += *b;
    return fmaxf(v, 0.f);
  }
};

template <bool VEC>
__device__ inline void spmm_epilogue(const SpmmArgs& a, int row, int col,
                                     typename Vec<VEC>::T acc) {
  using V = Vec<VEC>;
  float* dst = a.out + (int64_t)row * a.ld_out + col;
  if (a.epilogue == SPMM_BIAS_RELU) {
    acc = V::bias_relu(acc, a.bias ? a.bias + col : nullptr);
  } else if (a.epilogue == SPMM_ADD) {
    V::add(acc, V::load(a.res + (int64_t)row * a.ld_res + col));
  }
  V::store(dst, acc);
}

// One work item per group of G lanes; NC column vectors per lane per pass.
// Block b covers column slice b % nslices of the items of item block
// b / nslices.  With 8 slices, the blocks of one slice all run on one XCD
// (blocks are dispatched round-robin over the 8 XCDs), so each XCD gathers
// from its own n x sw slice of the input, which stays in that XCD's L2.
//
// The item's entries are taken in batches of G: each lane loads one index
// and value (a coalesced read), then the batch is walked with lane
// shuffles, eight neighbour rows in flight at a time, accumulating in entry
// order.  A 64-entry item thus costs a handful of memory round trips
// instead of one per entry.
constexpr int GATHER_DEPTH = 8;

template <int G, int NC, bool VEC>
__global__ __launch_bounds__(256) void spmm_items_kernel(SpmmArgs a) {
  using V = Vec<VEC>;
  using T = typename V::T;
  constexpr int IPB = 256 / G;
  constexpr int COLS = G * V::W * NC;
  const int slice = blockIdx.x % a.nslices;
  int item = (blockIdx.x / a.nslices) * IPB + threadIdx.x / G;
  if (G == 64) item = __builtin_amdgcn_readfirstlane(item);
  if (item >= a.hdr->n_items) return;
  const int4 it = a.items[item];
  const int row = it.x, b = it.y, e = it.z, slot = it.w;
  const int lane = threadIdx.x % G;
  const int c_lo = slice * a.sw;
  const int c_hi = min(a.w, c_lo + a.sw);
  const float* __restrict__ in = a.in;
  for (int c0 = c_lo; c0 < c_hi; c0 += COLS) {
    T acc[NC];
#pragma unroll
    for (int q = 0; q < NC; ++q) acc[q] = V::zero();
    for (int jb = b; jb < e; jb += G) {
      const int cnt = min(G, e - jb);
      const int my_idx = lane < cnt ? a.indices[jb + lane] : 0;
      const float my_val = lane < cnt ? a.vals[jb + lane] : 0.f;
      for (int k = 0; k < cnt; k += GATHER_DEPTH) {
        int idx[GATHER_DEPTH];
        float val[GATHER_DEPTH];
        T x[GATHER_DEPTH][NC];
#pragma unroll
        for (int u = 0; u < GATHER_DEPTH; ++u) {
          idx[u] = __shfl(my_idx, k + u, G);
          val[u] = __shfl(my_val, k + u, G);
        }
#pragma unroll
        for (int u = 0; u < GATHER_DEPTH; ++u)
#pragma unroll
          for (int q = 0; q < NC; ++q) {
            const int col = c0 + (q * G + lane) * V::W;
            x[u][q] = (k + u < cnt && col < c_hi)
                          ? V::load(in + (int64_t)idx[u] * a.ld_in + col)
                          : V::zero();
          }
#pragma unroll
        for (int u = 0; u < GATHER_DEPTH; ++u)
#pragma unroll
          for (int q = 0; q < NC; ++q)
            if (k + u < cnt) V::fma(acc[q], val[u], x[u][q]);
      }
    }
#pragma unroll
    for (int q = 0; q < NC; ++q) {
      const int col = c0 + (q * G + lane) * V::W;
      if (col < c_hi) {
        if (slot >= 0)
          V::store(a.part + (int64_t)slot * a.ldp + col, acc[q]);
        else
          spmm_epilogue<VEC>(a, row, col, acc[q]);
      }
    }
  }
}

// Sums the chunk partials of each split row in chunk order.
template <int G, int NC, bool VEC>
__global__ __launch_bounds__(256) void spmm_reduce_kernel(SpmmArgs a) {
  using V = Vec<VEC>;
  using T = typename V::T;
  constexpr int IPB = 256 / G;
  constexpr int COLS = G * V::W * NC;
  const int slice = blockIdx.x % a.nslices;
  int s = (blockIdx.x / a.nslices) * IPB + threadIdx.x / G;
  if (G == 64) s = __builtin_amdgcn_readfirstlane(s);
  if (s >= a.hdr->n_splits) return;
  const int4 sp = a.splits[s];
  const int row = sp.x, first = sp.y, cnt = sp.z;
  const int lane = threadIdx.x % G;
  const int c_lo = slice * a.sw;
  const int c_hi = min(a.w, c_lo + a.sw);
  for (int c0 = c_lo; c0 < c_hi; c0 += COLS) {
#pragma unroll
    for (int q = 0; q < NC; ++q) {
      const int col = c0 + (q * G + lane) * V::W;
      if (col < c_hi) {
        T acc = V::zero();
        const float* src = a.part + (int64_t)first * a.ldp + col;
        int k = 0;
        for (; k + 4 <= cnt; k += 4) {  // four partials in flight, added in order
          const T x0 = V::load(src + (int64_t)(k + 0) * a.ldp);
          const T x1 = V::load(src + (int64_t)(k + 1) * a.ldp);
          const T x2 = V::load(src + (int64_t)(k + 2) * a.ldp);
          const T x3 = V::load(src + (int64_t)(k + 3) * a.ldp);
          V::add(acc, x0);
          V::add(acc, x1);
          V::add(acc, x2);
          V::add(acc, x3);
        }
        for (; k < cnt; ++k) V::add(acc, V::load(src + (int64_t)k * a.ldp));
        spmm_epilogue<VEC>(a, row, col, acc);
      }
    }
  }
}

size_t spmm_partials_bytes(int32_t n, int64_t nnz, int32_t w) {
  const PlanDims d = plan_dims(n, nnz);
  if (d.max_slots == 0 || w <= 0) return 0;
  return round_up((size_t)d.max_slots * (size_t)round_up(w, 4) * 4, 256);
}

// Algorithmic bytes of one aggregation: row pointers, an index and a value
// per stored entry, the n x w input read once and the output written once.
static double spmm_bytes(int32_t n, int64_t nnz, int32_t w) {
  return 4.0 * (n + 1) + 8.0 * (double)nnz + 8.0 * (double)n * w;
}

template <int G, int NC, bool VEC>
static hipError_t spmm_run(const SpmmArgs& a, const PlanDims& d, int32_t n,
                           int64_t nnz, hipStream_t s) {
  constexpr int IPB = 256 / G;
  if (d.max_items > 0) {
    timer_begin(GNN_K_SPMM, s);
    spmm_items_kernel<G, NC, VEC>
        <<<(unsigned)(ceil_div(d.max_items, IPB) * a.nslices), 256, 0, s>>>(a);
    timer_end(GNN_K_SPMM, spmm_bytes(n, nnz, a.w), s);
  }
  if (d.max_splits > 0) {
    timer_begin(GNN_K_SPMM_REDUCE, s);
    spmm_reduce_kernel<G, NC, VEC>
        <<<(unsigned)(ceil_div(d.max_splits, IPB) * a.nslices), 256, 0, s>>>(a);
    timer_end(GNN_K_SPMM_REDUCE, 0.0, s);
  }
  return hipGetLastError();
}

template <bool VEC>
static hipError_t spmm_dispatch(const SpmmArgs& a, const PlanDims& d,
                                int32_t n, int64_t nnz, hipStream_t s) {
  const int units = VEC ? a.sw / 4 : a.sw;  // column vectors per slice row
  if (units <= 4) return spmm_run<4, 1, VEC>(a, d, n, nnz, s);
  if (units <= 8) return spmm_run<8, 1, VEC>(a, d, n, nnz, s);
  if (units <= 16) return spmm_run<16, 1, VEC>(a, d, n, nnz, s);
  if (units <= 32) return spmm_run<32, 1, VEC>(a, d, n, nnz, s);
  if (units <= 64) return spmm_run<64, 1, VEC>(a, d, n, nnz, s);
  if (units <= 128) return spmm_run<64, 2, VEC>(a, d, n, nnz, s);
  if (units <= 192) return spmm_run<64, 3, VEC>(a, d, n, nnz, s);
  return spmm_run<64, 4, VEC>(a, d, n, nnz, s);
}

hipError_t spmm_launch(const SpmmCall& c, hipStream_t s) {
  if (c.n <= 0 || c.w <= 0) return hipSuccess;
  const PlanDims d = plan_dims(c.n, c.nnz);
  const char* base = static_cast<const char*>(c.plan);
  SpmmArgs a;
  a.indices = c.indices;
  a.vals = c.vals;
  a.hdr = reinterpret_cast<const PlanHeader*>(base);
  a.items = reinterpret_cast<const int4*>(base + d.items_offset);
  a.splits = reinterpret_cast<const int4*>(base + d.splits_offset);
  a.w = c.w;
  a.in = c.in;
  a.ld_in = c.ld_in;
  a.out = c.out;
  a.ld_out = c.ld_out;
  a.epilogue = c.epilogue;
  a.bias = c.bias;
  a.res = c.res;
  a.ld_res = c.ld_res;
  a.part = c.partials;
  a.ldp = round_up(c.w, 4);
  // Wide rows are cut into 8 column slices, one per XCD (the GPU form of
  // the feature-column partition of Section 5.3, Theorem 2 / Algorithm 7,
  // with each XCD's L2 as the cache that a slice must fit).
  a.nslices = c.w >= 256 ? 8 : 1;
  a.sw = (int32_t)round_up(ceil_div(c.w, a.nslices), 4);
  const bool vec = (c.w % 4 == 0) && vec4_ok(c.in, c.ld_in) &&
                   vec4_ok(c.out, c.ld_out) &&
                   (c.epilogue != SPMM_BIAS_RELU || !c.bias || aligned16(c.bias)) &&
                   (c.epilogue != SPMM_ADD || vec4_ok(c.res, c.ld_res)) &&
                   (d.max_splits == 0 || aligned16(c.partials));
  return vec ? spmm_dispatch<true>(a, d, c.n, c.nnz, s)
             : spmm_dispatch<false>(a, d, c.n, c.nnz, s);
}

}  // namespace gnnprop
