// Sparse feature / gradient propagation on gfx950 (the first of the three
// kernels of Section 5.1) and the per-subgraph preparation it needs: the
// aggregation work plan and the transposed value array of Section 5.2
// (Algorithm 6).
//
// Aggregation design.  Row v of A_s . X is the weighted sum of the input
// rows of v's neighbours.  The stored entries are cut into windows of
// BLOCK_ENTRIES; workgroup i owns the rows whose first entry lies in window
// i (in windows 2i and 2i + 1 for large launches), i.e. a run of whole rows,
// so no row is shared between workgroups.  Its
// entry range is split evenly over its groups of G lanes; a group streams
// its entries (whatever their rows) with G-wide coalesced loads of index,
// value and row, then gathers the neighbour rows' feature columns as float4
// (D in flight) and accumulates in entry order, closing an output row
// whenever the row id changes.  A row cut between groups (power-law hubs
// span all of them) is finished through LDS by the group holding its first
// entry, adding the other groups' parts in group order.  One kernel, no
// atomics, bit-reproducible, and work is balanced by entries, not rows.
// Outputs of 32 columns and more are cut into 8 (or 16) column slices, each
// XCD gathering from its own (the GPU form of the feature partition of
// Section 5.3, Theorem 2 / Algorithm 7, with each XCD's L2 as the cache a
// slice should fit).
#include "internal.hpp"

namespace gnnprop {

// ------------------------------------------------------------- plan sizes

constexpr int BLOCK_ENTRIES = 256;

static int64_t plan_blocks(int64_t nnz) {
  return std::max<int64_t>(1, ceil_div(std::max<int64_t>(nnz, 0), BLOCK_ENTRIES));
}

PlanDims plan_dims(int32_t n, int64_t nnz) {
  (void)n;
  PlanDims d;
  d.block_entries = BLOCK_ENTRIES;
  d.nblk = plan_blocks(nnz);
  d.binfo_offset = round_up(sizeof(PlanHeader), 256);
  d.erow_offset = round_up(d.binfo_offset + 16 * (size_t)d.nblk, 256);
  d.bytes = round_up(d.erow_offset + 4 * (size_t)std::max<int64_t>(nnz, 0), 256);
  return d;
}

// ----------------------------------------------------------- plan build
//
// Workgroup k owns rows [r_lo(k), r_lo(k+1)) with r_lo(k) the first row
// whose first entry is at or after k * BLOCK_ENTRIES (the last one also
// owns the trailing empty rows).  Row r is r_lo(k) exactly for the window
// starts in (indptr[r-1], indptr[r]], so one thread per row writes them
// without any scan.  A second kernel writes each entry's row.

__global__ __launch_bounds__(256) void plan_blocks_kernel(
    const int32_t* __restrict__ indptr, int32_t n, int64_t nnz,
    int32_t nblk, int4* __restrict__ binfo, PlanHeader* __restrict__ hdr) {
  const int r = blockIdx.x * 256 + threadIdx.x;
  if (r > n) return;
  const int p = indptr[r];
  const int k_lo = r == 0 ? 0 : indptr[r - 1] / BLOCK_ENTRIES + 1;
  const int k_hi = min(p / BLOCK_ENTRIES, nblk - 1);
  for (int k = k_lo; k <= k_hi; ++k) {
    binfo[k].x = r;
    binfo[k].z = p;
    if (k > 0) {
      binfo[k - 1].y = r;
      binfo[k - 1].w = p;
    }
  }
  if (r == n) {
    binfo[nblk - 1].y = n;
    binfo[nblk - 1].w = (int)nnz;
    PlanHeader h;
    memset(&h, 0, sizeof(h));
    h.nblk = nblk;
    h.block_entries = BLOCK_ENTRIES;
    h.n = n;
    h.nnz = (int)nnz;
    *hdr = h;
  }
}

// Row of every entry; one wavefront per row.
__global__ __launch_bounds__(256) void plan_rows_kernel(
    const int32_t* __restrict__ indptr, int32_t n,
    int32_t* __restrict__ erow) {
  const int r = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (r >= n) return;
  const int lane = threadIdx.x & 63;
  const int b = indptr[r], e = indptr[r + 1];
  for (int j = b + lane; j < e; j += 64) erow[j] = r;
}

hipError_t plan_build_launch(int32_t n, int64_t nnz, const int32_t* indptr,
                             const int32_t* indices, void* plan,
                             hipStream_t s) {
  (void)indices;
  const PlanDims d = plan_dims(n, nnz);
  char* base = static_cast<char*>(plan);
  timer_begin(GNN_K_PLAN, s);
  plan_blocks_kernel<<<(unsigned)ceil_div((int64_t)n + 1, 256), 256, 0, s>>>(
      indptr, n, nnz, (int32_t)d.nblk,
      reinterpret_cast<int4*>(base + d.binfo_offset),
      reinterpret_cast<PlanHeader*>(base));
  if (n > 0 && nnz > 0)
    plan_rows_kernel<<<(unsigned)ceil_div(n, 4), 256, 0, s>>>(
        indptr, n, reinterpret_cast<int32_t*>(base + d.erow_offset));
  timer_end(GNN_K_PLAN, 8.0 * (n + 1) + 4.0 * nnz, s);
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

// One thread per entry, its row taken from the plan, so that a hub row is
// spread over as many threads as it has entries.
__global__ __launch_bounds__(256) void transpose_values_entries_kernel(
    int64_t nnz, const int32_t* __restrict__ erow,
    const int32_t* __restrict__ indptr, const int32_t* __restrict__ indices,
    const float* __restrict__ vals, float* __restrict__ vals_t) {
  const int64_t j = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (j >= nnz) return;
  transpose_entry(erow[j], (int)j, indptr, indices, vals, vals_t);
}

hipError_t transpose_values_launch(int32_t n, int64_t nnz,
                                   const int32_t* indptr,
                                   const int32_t* indices, const float* vals,
                                   float* vals_t, const void* plan,
                                   hipStream_t s) {
  if (n <= 0 || nnz <= 0) return hipSuccess;
  timer_begin(GNN_K_TRANSPOSE, s);
  if (plan) {
    const PlanDims d = plan_dims(n, nnz);
    const char* base = static_cast<const char*>(plan);
    transpose_values_entries_kernel<<<(unsigned)ceil_div(nnz, 256), 256, 0, s>>>(
        nnz, reinterpret_cast<const int32_t*>(base + d.erow_offset), indptr,
        indices, vals, vals_t);
  } else {
    transpose_values_kernel<<<(unsigned)ceil_div(n, 4), 256, 0, s>>>(
        n, indptr, indices, vals, vals_t);
  }
  timer_end(GNN_K_TRANSPOSE, 0.0, s);
  return hipGetLastError();
}

// ------------------------------------------ plan + transposed values, fused
//
// Both per-subgraph preparations in one launch.  Blocks [0, nrow_blocks)
// write the window records (one thread per row, as plan_blocks_kernel);
// the others take 256 consecutive entries each: the block's first thread
// finds the rows holding its first and last entry by binary search over
// indptr, then every thread finds its own entry's row between those two
// (a few steps), writes it to the plan and moves its value to the transposed
// position (transpose_entry).  The two halves write disjoint parts of the
// plan.
__global__ __launch_bounds__(256) void prepare_kernel(
    const int32_t* __restrict__ indptr, const int32_t* __restrict__ indices,
    const float* __restrict__ vals, float* __restrict__ vals_t, int32_t n,
    int64_t nnz, int32_t nblk, int32_t nrow_blocks, int4* __restrict__ binfo,
    PlanHeader* __restrict__ hdr, int32_t* __restrict__ erow) {
  if ((int)blockIdx.x < nrow_blocks) {
    const int r = blockIdx.x * 256 + threadIdx.x;
    if (r > n) return;
    const int p = indptr[r];
    const int k_lo = r == 0 ? 0 : indptr[r - 1] / BLOCK_ENTRIES + 1;
    const int k_hi = min(p / BLOCK_ENTRIES, nblk - 1);
    for (int k = k_lo; k <= k_hi; ++k) {
      binfo[k].x = r;
      binfo[k].z = p;
      if (k > 0) {
        binfo[k - 1].y = r;
        binfo[k - 1].w = p;
      }
    }
    if (r == n) {
      binfo[nblk - 1].y = n;
      binfo[nblk - 1].w = (int)nnz;
      PlanHeader h;
      memset(&h, 0, sizeof(h));
      h.nblk = nblk;
      h.block_entries = BLOCK_ENTRIES;
      h.n = n;
      h.nnz = (int)nnz;
      *hdr = h;
    }
    return;
  }
  // the last row r with indptr[r] <= j, searched in [lo, hi]
  auto row_of = [&](int j, int lo, int hi) {
    while (lo < hi) {
      const int mid = (lo + hi + 1) >> 1;
      if (indptr[mid] <= j)
        lo = mid;
      else
        hi = mid - 1;
    }
    return lo;
  };
  const int64_t j0 = (int64_t)(blockIdx.x - nrow_blocks) * 256;
  const int64_t j1 = min<int64_t>(j0 + 256, nnz) - 1;
  // Rows of the block's first and last entry by a 128-way search each
  // (threads 0-127 for j0, 128-255 for j1): every round probes 128 evenly
  // spaced row starts at once and keeps the chunk holding the answer, so
  // the chain of dependent loads is log_128 n long instead of log_2 n.
  __shared__ int cnt[2], lo_s[2], hi_s[2];
  const int half = threadIdx.x >> 7, t = threadIdx.x & 127;
  const int jj = (int)(half ? j1 : j0);
  int rounds = 0;
  for (int64_t sz = n; sz > 1; sz = (sz + 127) / 128) ++rounds;
  if (t == 0) {
    lo_s[half] = 0;
    hi_s[half] = n - 1;
  }
  for (int rd = 0; rd < rounds; ++rd) {
    if (t == 0) cnt[half] = 0;
    __syncthreads();
    const int lo = lo_s[half], hi = hi_s[half];
    const int c = (hi - lo + 128) / 128;  // chunk: ceil((hi - lo + 1) / 128)
    const int pos = lo + t * c;
    if (pos <= hi && indptr[pos] <= jj) atomicAdd(&cnt[half], 1);
    __syncthreads();
    if (t == 0) {
      const int T = cnt[half];  // >= 1: indptr[lo] <= jj always holds
      lo_s[half] = lo + (T - 1) * c;
      hi_s[half] = min(hi, lo + T * c - 1);
    }
  }
  __syncthreads();
  __shared__ int bounds[2];
  if (threadIdx.x == 0) {
    bounds[0] = lo_s[0];
    bounds[1] = lo_s[1];
  }
  __syncthreads();
  const int64_t j = j0 + threadIdx.x;
  if (j > j1) return;
  const int v = row_of((int)j, bounds[0], bounds[1]);
  erow[j] = v;
  transpose_entry(v, (int)j, indptr, indices, vals, vals_t);
}

hipError_t prepare_launch(int32_t n, int64_t nnz, const int32_t* indptr,
                          const int32_t* indices, const float* vals,
                          float* vals_t, void* plan, hipStream_t s) {
  const PlanDims d = plan_dims(n, nnz);
  char* base = static_cast<char*>(plan);
  const int rb = (int)ceil_div((int64_t)n + 1, 256);
  const int eb = (n > 0 && nnz > 0) ? (int)ceil_div(nnz, 256) : 0;
  timer_begin(GNN_K_PLAN, s);
  prepare_kernel<<<(unsigned)(rb + eb), 256, 0, s>>>(
      indptr, indices, vals, vals_t, n, nnz, (int32_t)d.nblk, rb,
      reinterpret_cast<int4*>(base + d.binfo_offset),
      reinterpret_cast<PlanHeader*>(base),
      reinterpret_cast<int32_t*>(base + d.erow_offset));
  timer_end(GNN_K_PLAN, 8.0 * (n + 1) + 16.0 * nnz, s);
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
  const int32_t* indptr;
  const int32_t* indices;
  const float* vals;
  const int4* binfo;   // per workgroup: rows [x, y), entries [z, w)
  const int32_t* erow;
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
  int32_t nslices;  // column slices: 1, or a multiple of 8
  int32_t sw;       // slice width in columns
  int32_t nwin;     // workgroups per slice: plan windows / wpb, rounded up
  int32_t wpb;      // consecutive plan windows per workgroup (1 or 2)
  int32_t nblk;     // plan windows
  int32_t weights;  // SpmmWeights
};

// Column slices.  Blocks are dispatched round-robin over the 8 XCDs, so with
// S = 8 P slices, block b = p (8 nwin) + 8 win + x works on slice 8 p + x of
// window (group) win: XCD x gathers only from slices x, x + 8, ..., one pass after
// the other, and each n x sw slice is sized to stay in that XCD's L2 (the
// cache-sized feature partitions of Theorem 2 / Algorithm 7).
//
// A group of G lanes covers G * W consecutive columns of the slice per pass
// (W = 4: float4 per lane, so one gathered 256-byte row segment of a
// 64-column slice is one quarter of a wavefront's load instruction, the
// widest access a lane has).  The group's entries are taken in batches of G
// (one coalesced index / value / row load per lane, the next batch
// prefetched), walked with lane shuffles, D neighbour rows in flight.  EPI
// is the epilogue; OFF32 marks inputs below 4 GiB, whose gather offsets fit
// 32 bits.
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
  // output rows are stored nontemporal: written once, read by the next
  // kernel, they would otherwise take L2 lines from the gathered rows
  __device__ static void store(float* p, T v) {
    typedef float f4v __attribute__((ext_vector_type(4)));
    const f4v x = {v.x, v.y, v.z, v.w};
    __builtin_nontemporal_store(x, reinterpret_cast<f4v*>(p));
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
  __device__ static void scale(T& acc, float s) {
    acc.x *= s;
    acc.y *= s;
    acc.z *= s;
    acc.w *= s;
  }
  __device__ static T relu(T v) {
    v.x = fmaxf(v.x, 0.f);
    v.y = fmaxf(v.y, 0.f);
    v.z = fmaxf(v.z, 0.f);
    v.w = fmaxf(v.w, 0.f);
    return v;
  }
  // the first k (1..3) components only: the ragged end of a row whose width
  // is not a multiple of 4
  __device__ static T load_part(const float* p, int k) {
    T v = zero();
    v.x = p[0];
    if (k > 1) v.y = p[1];
    if (k > 2) v.z = p[2];
    return v;
  }
  __device__ static void store_part(float* p, T v, int k) {
    p[0] = v.x;
    if (k > 1) p[1] = v.y;
    if (k > 2) p[2] = v.z;
  }
  // rounded to bf16: all four values, or the first k (1..3)
  __device__ static void store_h(uint16_t* p, T v) {
    *reinterpret_cast<uint2*>(p) = make_uint2(pack_bf16(v.x, v.y), pack_bf16(v.z, v.w));
  }
  __device__ static void store_h_part(uint16_t* p, T v, int k) {
    const uint32_t a = pack_bf16(v.x, v.y), b = pack_bf16(v.z, v.w);
    p[0] = (uint16_t)(a & 0xffffu);
    if (k > 1) p[1] = (uint16_t)(a >> 16);
    if (k > 2) p[2] = (uint16_t)(b & 0xffffu);
  }
  // v where m > 0, else 0 (a selection: NaN or infinite v is not spread)
  __device__ static T select_pos(T m, T v) {
    v.x = m.x > 0.f ? v.x : 0.f;
    v.y = m.y > 0.f ? v.y : 0.f;
    v.z = m.z > 0.f ? v.z : 0.f;
    v.w = m.w > 0.f ? v.w : 0.f;
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
  __device__ static void scale(T& acc, float s) { acc *= s; }
  __device__ static T relu(T v) { return fmaxf(v, 0.f); }
  __device__ static T select_pos(T m, T v) { return m > 0.f ? v : 0.f; }
  __device__ static T load_part(const float* p, int) { return *p; }
  __device__ static void store_part(float* p, T v, int) { *p = v; }
  __device__ static void store_h(uint16_t* p, T v) { *p = (uint16_t)(pack_bf16(v, 0.f) & 0xffffu); }
  __device__ static void store_h_part(uint16_t* p, T v, int) { store_h(p, v); }
};

template <int G, int D, bool VEC, int EPI, bool OFF32, bool RAG>
__global__ __launch_bounds__(256) void spmm_kernel(SpmmArgs a) {
  using V = Vec<VEC>;
  using T = typename V::T;
  constexpr int EMPTY = -2;     // group range holds no entry
  // Lane groups: G consecutive lanes of a wavefront (1 <= G <= 64), 64 / G
  // groups per wavefront (the lanes past the last group take no part),
  // groups numbered wavefront by wavefront.  A group's lane l is thread
  // gtid(g) + l, so the per-lane LDS slots are indexed by thread.
  constexpr int gpw = 64 / G;   // groups per wavefront
  constexpr int NG = 4 * gpw;   // groups per block
  constexpr int CW = G * V::W;  // columns per pass
  __shared__ T head[256];       // part of a row begun in an earlier group
  __shared__ T tail[256];       // part of a row that goes on past the group
  __shared__ int head_row[256], tail_row[256], starts[256];
  auto gtid = [&](int g) { return (g / gpw) * 64 + (g % gpw) * G; };

  int slice = 0, win = blockIdx.x;
  if (a.nslices >= 8) {
    const int per = 8 * a.nwin;
    const int r = (int)(blockIdx.x % per);
    slice = 8 * (int)(blockIdx.x / per) + (r & 7);
    win = r >> 3;
  }
  // Consecutive windows own consecutive rows and entries (an empty window
  // inside a hub row starts and ends where the next row starts), so
  // windows k .. k + wpb - 1 together are one run of whole rows.
  const int k0 = win * a.wpb, k1 = min(k0 + a.wpb, a.nblk) - 1;
  const int4 bi0 = a.binfo[k0], bi1 = a.binfo[k1];
  const int r_lo = bi0.x, r_hi = bi1.y, B = bi0.z, E = bi1.w;
  const int tid = threadIdx.x;
  const int wl = tid & 63, lg = wl / G;
  const bool member = lg < gpw;            // lane belongs to a group
  const int gi = (tid >> 6) * gpw + lg;    // group id (member lanes)
  const int lane = wl - lg * G;            // lane within the group
  const int base = lg * G;                 // the group's first lane in the wavefront
  const int gb = member ? B + (int)((int64_t)(E - B) * gi / NG) : 0;
  const int ge = member ? B + (int)((int64_t)(E - B) * (gi + 1) / NG) : 0;
  const int c_lo = slice * a.sw;
  const int c_hi = min(a.w, c_lo + a.sw);
  const float* __restrict__ in = a.in;
  const int32_t* __restrict__ indices = a.indices;
  const int32_t* __restrict__ erow = a.erow;
  const float* __restrict__ vals = a.vals;
  const uint32_t ld_in = (uint32_t)a.ld_in;
  const int32_t* __restrict__ indptr = a.indptr;
  const int wmode = a.weights;
  // weight of stored entry j (column idx); see SpmmWeights
  auto weight = [&](int j, int idx) -> float {
    if (wmode == SPMM_W_VALUES) return vals[j];
    if (wmode == SPMM_W_ROW_SCALE) return 1.f;
    const int d = indptr[idx + 1] - indptr[idx];
    return d > 0 ? 1.f / (float)d : 0.f;
  };

  // rows of the entries just outside this group's range (-1: none)
  int prev_row = -1, next_row = -1;
  if (gb < ge) {
    if (gb > B) prev_row = erow[gb - 1];
    if (ge < E) next_row = erow[ge];
  }

  for (int c0 = c_lo; c0 < c_hi; c0 += CW) {
    const int col = c0 + lane * V::W;
    const bool ok = member && col < c_hi;
    // a lane holding the ragged end of the row (fewer than W columns left)
    const int nv = c_hi - col;
    const bool part = RAG && ok && nv < V::W;
    auto ld = [&](const float* p) { return part ? V::load_part(p, nv) : V::load(p); };
    auto finish = [&](int row, T acc) {
      if (!ok) return;
      if (wmode == SPMM_W_ROW_SCALE)  // a row with entries: deg >= 1
        V::scale(acc, 1.f / (float)(indptr[row + 1] - indptr[row]));
      if (EPI == SPMM_BIAS_RELU) {
        if (a.bias) V::add(acc, ld(a.bias + col));
        acc = V::relu(acc);
      } else if (EPI == SPMM_ADD) {
        V::add(acc, ld(a.res + (int64_t)row * a.ld_res + col));
        if (a.mask) acc = V::select_pos(ld(a.mask + (int64_t)row * a.ld_mask + col), acc);
      }
      if (EPI == SPMM_STORE_BF16) {
        uint16_t* dst = reinterpret_cast<uint16_t*>(a.out) + (int64_t)row * a.ld_out + col;
        if (part)
          V::store_h_part(dst, acc, nv);
        else
          V::store_h(dst, acc);
        return;
      }
      float* dst = a.out + (int64_t)row * a.ld_out + col;
      if (part)
        V::store_part(dst, acc, nv);
      else
        V::store(dst, acc);
    };

    int hr = EMPTY, tr = -1, nstart = 0;
    if (gb < ge) {
      hr = -1;
      int cur = -1, first_row = -1;
      T acc = V::zero();
      // A closed row is written out unless part of it lies in another
      // group: then it goes to LDS for the group holding its first entry.
      auto close = [&](bool last) {
        const bool opened_before = cur == first_row && prev_row == cur;
        const bool goes_on = last && next_row == cur;
        if (goes_on && !opened_before) {
          tail[tid] = acc;
          tr = cur;
        } else if (opened_before) {
          head[tid] = acc;
          hr = cur;
        } else {
          finish(cur, acc);
        }
      };
      int ni = 0, nr = 0;
      float nv = 0.f;
      if (lane < ge - gb) {
        ni = indices[gb + lane];
        nv = weight(gb + lane, ni);
        nr = erow[gb + lane];
      }
      for (int jb = gb; jb < ge; jb += G) {
        const int cnt = min(G, ge - jb);
        const int fi = ni, fr = nr;
        const float fv = nv;
        if (jb + G < ge) {  // prefetch the next batch
          const int j2 = jb + G + lane;
          const bool in_r = j2 < ge;
          ni = in_r ? indices[j2] : 0;
          nv = in_r ? weight(j2, ni) : 0.f;
          nr = in_r ? erow[j2] : 0;
        }
        for (int k = 0; k < cnt; k += D) {
          T x[D];
#pragma unroll
          for (int u = 0; u < D; ++u) {
            const int idx = __shfl(fi, base + k + u);
            if (k + u < cnt && ok) {
              if (OFF32)
                x[u] = ld(reinterpret_cast<const float*>(
                    reinterpret_cast<const char*>(in) +
                    (((uint32_t)idx * ld_in + (uint32_t)col) << 2)));
              else
                x[u] = ld(in + (int64_t)idx * a.ld_in + col);
            } else {
              x[u] = V::zero();
            }
          }
#pragma unroll
          for (int u = 0; u < D; ++u) {
            if (k + u < cnt) {
              const int rw = __shfl(fr, base + k + u);
              const float val = __shfl(fv, base + k + u);
              if (rw != cur) {
                if (cur >= 0) close(false);
                if (cur < 0) first_row = rw;
                cur = rw;
                nstart += (cur == first_row && prev_row == cur) ? 0 : 1;
                acc = V::zero();
              }
              V::fma(acc, val, x[u]);
            }
          }
        }
      }
      close(true);
    }
    if (member && lane == 0) {
      head_row[gi] = hr;
      tail_row[gi] = tr;
      starts[gi] = nstart;
    }
    __syncthreads();
    if (tr >= 0) {  // this group holds the first entry of a shared row
      T s = tail[tid];
      for (int g = gi + 1; g < NG; ++g) {
        const int h = head_row[g];
        if (h == EMPTY) continue;
        if (h != tr) break;
        V::add(s, head[gtid(g) + lane]);
      }
      finish(tr, s);
    }
    // Rows without entries get the epilogue of a zero sum.
    int owned = 0;
    for (int g = 0; g < NG; ++g) owned += starts[g];
    if (owned < r_hi - r_lo) {
      for (int r = r_lo + tid; r < r_hi; r += 256) {
        if (a.indptr[r] == a.indptr[r + 1]) {
          for (int c = c0; c < min(c_hi, c0 + CW); ++c) {
            float v = 0.f;
            if (EPI == SPMM_BIAS_RELU) {
              v = fmaxf(a.bias ? a.bias[c] : 0.f, 0.f);
            } else if (EPI == SPMM_ADD) {
              v = a.res[(int64_t)r * a.ld_res + c];
              if (a.mask && !(a.mask[(int64_t)r * a.ld_mask + c] > 0.f)) v = 0.f;
            }
            if (EPI == SPMM_STORE_BF16)
              reinterpret_cast<uint16_t*>(a.out)[(int64_t)r * a.ld_out + c] = 0;
            else
              a.out[(int64_t)r * a.ld_out + c] = v;
          }
        }
      }
    }
    __syncthreads();
  }
}

// Gather floor.  The aggregation's own loads in its own order, and nothing
// else: the same grid, column slices, lane groups, entry ranges, batches of
// G index / value loads and D gathers in flight, but one accumulator per
// lane for all of the group's entries instead of one per row, no entry rows
// read, no row closing and no LDS finish of shared rows.  The block's total
// per column (summed over its groups in group order) is written to the
// window's first row and zeros to its other rows, so that every output row
// is still written once and the column sums of `out` equal those of
// A_s . in.  Its time is what this gather order costs on the chip: the
// floor against which the aggregation's own bookkeeping is measured.
template <int G, int D, bool OFF32, bool RAG>
__global__ __launch_bounds__(256) void spmm_floor_kernel(SpmmArgs a) {
  using V = Vec<true>;
  using T = typename V::T;
  constexpr int gpw = 64 / G;
  constexpr int NG = 4 * gpw;
  constexpr int CW = G * V::W;
  __shared__ T part[256];
  auto gtid = [&](int g) { return (g / gpw) * 64 + (g % gpw) * G; };

  int slice = 0, win = blockIdx.x;
  if (a.nslices >= 8) {
    const int per = 8 * a.nwin;
    const int r = (int)(blockIdx.x % per);
    slice = 8 * (int)(blockIdx.x / per) + (r & 7);
    win = r >> 3;
  }
  const int k0 = win * a.wpb, k1 = min(k0 + a.wpb, a.nblk) - 1;
  const int4 bi0 = a.binfo[k0], bi1 = a.binfo[k1];
  const int r_lo = bi0.x, r_hi = bi1.y, B = bi0.z, E = bi1.w;
  const int tid = threadIdx.x;
  const int wl = tid & 63, lg = wl / G;
  const bool member = lg < gpw;
  const int gi = (tid >> 6) * gpw + lg;
  const int lane = wl - lg * G;
  const int base = lg * G;
  const int gb = member ? B + (int)((int64_t)(E - B) * gi / NG) : 0;
  const int ge = member ? B + (int)((int64_t)(E - B) * (gi + 1) / NG) : 0;
  const int c_lo = slice * a.sw;
  const int c_hi = min(a.w, c_lo + a.sw);
  const float* __restrict__ in = a.in;
  const int32_t* __restrict__ indices = a.indices;
  const float* __restrict__ vals = a.vals;
  const uint32_t ld_in = (uint32_t)a.ld_in;

  for (int c0 = c_lo; c0 < c_hi; c0 += CW) {
    const int col = c0 + lane * V::W;
    const bool ok = member && col < c_hi;
    const int nv = c_hi - col;
    const bool prt = RAG && ok && nv < V::W;
    auto ld = [&](const float* p) { return prt ? V::load_part(p, nv) : V::load(p); };
    T acc = V::zero();
    int ni = 0;
    float nw = 0.f;
    if (gb < ge && lane < ge - gb) {
      ni = indices[gb + lane];
      nw = vals[gb + lane];
    }
    for (int jb = gb; jb < ge; jb += G) {
      const int cnt = min(G, ge - jb);
      const int fi = ni;
      const float fv = nw;
      if (jb + G < ge) {
        const int j2 = jb + G + lane;
        const bool in_r = j2 < ge;
        ni = in_r ? indices[j2] : 0;
        nw = in_r ? vals[j2] : 0.f;
      }
      for (int k = 0; k < cnt; k += D) {
        T x[D];
#pragma unroll
        for (int u = 0; u < D; ++u) {
          const int idx = __shfl(fi, base + k + u);
          if (k + u < cnt && ok) {
            if (OFF32)
              x[u] = ld(reinterpret_cast<const float*>(
                  reinterpret_cast<const char*>(in) +
                  (((uint32_t)idx * ld_in + (uint32_t)col) << 2)));
            else
              x[u] = ld(in + (int64_t)idx * a.ld_in + col);
          } else {
            x[u] = V::zero();
          }
        }
#pragma unroll
        for (int u = 0; u < D; ++u) {
          const float val = __shfl(fv, base + k + u);
          if (k + u < cnt) V::fma(acc, val, x[u]);
        }
      }
    }
    part[tid] = acc;
    __syncthreads();
    if (member) {
      for (int r = r_lo + gi; r < r_hi; r += NG) {
        T v = V::zero();
        if (r == r_lo)
          for (int g = 0; g < NG; ++g) V::add(v, part[gtid(g) + lane]);
        if (ok) {
          float* dst = a.out + (int64_t)r * a.ld_out + col;
          if (prt)
            V::store_part(dst, v, nv);
          else
            V::store(dst, v);
        }
      }
    }
    __syncthreads();
  }
}

// Algorithmic bytes of one aggregation: row pointers, an index and a value
// per stored entry, the n x w input read once and the output written once.
static double spmm_bytes(int32_t n, int64_t nnz, int32_t w, int out_bytes = 4) {
  return 4.0 * (n + 1) + 8.0 * (double)nnz + (4.0 + out_bytes) * (double)n * w;
}

#ifndef SPMM_DEPTH
#define SPMM_DEPTH 4
#endif

template <int G, bool VEC, int EPI, bool RAG>
static void spmm_go(const SpmmArgs& a, bool off32, hipStream_t s) {
  const unsigned grid = (unsigned)((int64_t)a.nwin * a.nslices);
  if (off32)
    spmm_kernel<G, SPMM_DEPTH, VEC, EPI, true, RAG><<<grid, 256, 0, s>>>(a);
  else
    spmm_kernel<G, SPMM_DEPTH, VEC, EPI, false, RAG><<<grid, 256, 0, s>>>(a);
}

template <int G, bool VEC, bool RAG>
static void spmm_epi(const SpmmArgs& a, bool off32, hipStream_t s) {
  switch (a.epilogue) {
    case SPMM_BIAS_RELU: return spmm_go<G, VEC, SPMM_BIAS_RELU, RAG>(a, off32, s);
    case SPMM_ADD: return spmm_go<G, VEC, SPMM_ADD, RAG>(a, off32, s);
    case SPMM_STORE_BF16:  // aligned rows only (spmm_launch checks)
      if constexpr (VEC) return spmm_go<G, VEC, SPMM_STORE_BF16, RAG>(a, off32, s);
      return;
    default: return spmm_go<G, VEC, SPMM_STORE, RAG>(a, off32, s);
  }
}

// Lane group width for a slice row of `units` float4s (or floats): a power
// of two covering it, or 10 lanes for the 10-unit rows of 8 slices (300
// columns: six groups to a wavefront instead of four 16-lane groups with 6
// idle lanes each, 8,000 x 300 aggregation 39.6 -> 35.8 us; with 16 slices,
// 602 columns, 16 lanes stay faster: 44.4 against 45.8 us).  RAG: float4
// lanes on a width that is not a multiple of 4 (the lane at the row's end
// reads and writes its 1..3 columns one by one).
template <bool VEC, bool RAG>
static void spmm_dispatch(const SpmmArgs& a, bool off32, hipStream_t s) {
  const int units = VEC ? ceil_div(a.sw, 4) : a.sw;  // column vectors per slice row
  if (units <= 4) return spmm_epi<4, VEC, RAG>(a, off32, s);
  if (units <= 8) return spmm_epi<8, VEC, RAG>(a, off32, s);
  if (units == 10 && a.nslices == 8) return spmm_epi<10, VEC, RAG>(a, off32, s);
  if (units <= 16) return spmm_epi<16, VEC, RAG>(a, off32, s);
  if (units <= 32) return spmm_epi<32, VEC, RAG>(a, off32, s);
  return spmm_epi<64, VEC, RAG>(a, off32, s);
}

size_t spmm_partials_bytes(int32_t n, int64_t nnz, int32_t w) {
  (void)n;
  (void)nnz;
  (void)w;
  return 0;
}

// Launch arguments of an aggregation call: column slices, lane groups and
// windows per workgroup; *vec: float4 lanes possible, *off32: 32-bit
// gather offsets.
static SpmmArgs spmm_args(const SpmmCall& c, bool* vec_out, bool* off32_out) {
  const PlanDims d = plan_dims(c.n, c.nnz);
  const char* base = static_cast<const char*>(c.plan);
  SpmmArgs a;
  memset(&a, 0, sizeof(a));
  a.indptr = c.indptr;
  a.indices = c.indices;
  a.vals = c.vals;
  a.binfo = reinterpret_cast<const int4*>(base + d.binfo_offset);
  a.erow = reinterpret_cast<const int32_t*>(base + d.erow_offset);
  a.w = c.w;
  a.in = c.in;
  a.ld_in = c.ld_in;
  a.out = c.out;
  a.ld_out = c.ld_out;
  a.epilogue = c.epilogue;
  a.bias = c.bias;
  a.res = c.res;
  a.ld_res = c.ld_res;
  a.mask = c.mask;
  a.ld_mask = c.ld_mask;
  a.weights = c.weights;
  // 8 slices (one per XCD) from 32 columns up.  A lane group covers the
  // float4 columns of a slice row (spmm_dispatch); when 8 slices need
  // groups of more than 16 lanes with over a quarter of them idle (602
  // columns: 76-column slices on 32 lanes), 16 slices are faster, having
  // twice the groups, and so the gathers, in flight per block.
  a.nslices = c.w >= 32 ? 8 : 1;
  a.sw = (int32_t)round_up(ceil_div(c.w, a.nslices), 4);
  if (a.nslices == 8 && a.sw > 64) {
    const int units = a.sw / 4;
    int g = 1;
    while (g < units) g *= 2;
    if (4 * units < 3 * g) {
      a.nslices = 16;
      a.sw = (int32_t)round_up(ceil_div(c.w, a.nslices), 4);
    }
  }
  // Two windows per workgroup once the grid would pass 16,384 workgroups:
  // each workgroup pays a chain of dependent loads (window record, entry
  // metadata, first gathers) before its gathers stream, which a longer entry
  // range amortises (50,000 nodes x 256 columns: 213 -> 175 us; 20,000 x
  // 200: 80 -> 77 us); smaller launches keep one (8,000 x 512: even).
  a.nblk = (int32_t)d.nblk;
  a.wpb = d.nblk * a.nslices > 16384 ? 2 : 1;
  a.nwin = (int32_t)ceil_div(d.nblk, (int64_t)a.wpb);
  // float4 lanes whenever rows start 16-byte aligned (the ragged end of a
  // width that is not a multiple of 4 is read and written per component)
  const bool out_ok = c.epilogue == SPMM_STORE_BF16
                          ? (reinterpret_cast<uintptr_t>(c.out) % 8 == 0 && c.ld_out % 4 == 0)
                          : vec4_ok(c.out, c.ld_out);
  const bool vec = vec4_ok(c.in, c.ld_in) && out_ok &&
                   (c.epilogue != SPMM_BIAS_RELU || !c.bias || aligned16(c.bias)) &&
                   (c.epilogue != SPMM_ADD || vec4_ok(c.res, c.ld_res)) &&
                   (!c.mask || vec4_ok(c.mask, c.ld_mask));
  // Gather offsets in 32 bits when the input spans less than 4 GiB.
  const bool off32 = ((int64_t)(c.n - 1) * c.ld_in + c.w) * 4 < (int64_t(1) << 32);
  *vec_out = vec;
  *off32_out = off32;
  return a;
}

hipError_t spmm_launch(const SpmmCall& c, hipStream_t s) {
  if (c.n <= 0 || c.w <= 0) return hipSuccess;
  bool vec = false, off32 = false;
  const SpmmArgs a = spmm_args(c, &vec, &off32);
  if (c.epilogue == SPMM_STORE_BF16 && !vec) return hipErrorInvalidValue;
  timer_begin(GNN_K_SPMM, s);
  if (vec && c.w % 4 != 0)
    spmm_dispatch<true, true>(a, off32, s);
  else if (vec)
    spmm_dispatch<true, false>(a, off32, s);
  else
    spmm_dispatch<false, false>(a, off32, s);
  timer_end(GNN_K_SPMM, spmm_bytes(c.n, c.nnz, c.w, c.epilogue == SPMM_STORE_BF16 ? 2 : 4), s);
  return hipGetLastError();
}

template <int G, bool RAG>
static void spmm_floor_go(const SpmmArgs& a, bool off32, hipStream_t s) {
  const unsigned grid = (unsigned)((int64_t)a.nwin * a.nslices);
  if (off32)
    spmm_floor_kernel<G, SPMM_DEPTH, true, RAG><<<grid, 256, 0, s>>>(a);
  else
    spmm_floor_kernel<G, SPMM_DEPTH, false, RAG><<<grid, 256, 0, s>>>(a);
}

template <bool RAG>
static void spmm_floor_dispatch(const SpmmArgs& a, bool off32, hipStream_t s) {
  const int units = ceil_div(a.sw, 4);  // the lane groups of spmm_dispatch
  if (units <= 4) return spmm_floor_go<4, RAG>(a, off32, s);
  if (units <= 8) return spmm_floor_go<8, RAG>(a, off32, s);
  if (units == 10 && a.nslices == 8) return spmm_floor_go<10, RAG>(a, off32, s);
  if (units <= 16) return spmm_floor_go<16, RAG>(a, off32, s);
  if (units <= 32) return spmm_floor_go<32, RAG>(a, off32, s);
  return spmm_floor_go<64, RAG>(a, off32, s);
}

hipError_t spmm_floor_launch(const SpmmCall& c, hipStream_t s) {
  if (c.n <= 0 || c.w <= 0) return hipSuccess;
  bool vec = false, off32 = false;
  const SpmmArgs a = spmm_args(c, &vec, &off32);
  if (!vec) return hipErrorInvalidValue;
  if (c.w % 4 != 0)
    spmm_floor_dispatch<true>(a, off32, s);
  else
    spmm_floor_dispatch<false>(a, off32, s);
  return hipGetLastError();
}

}  // namespace gnnprop
