// Subgraph preparation on the GPU: the subgraph of the full training graph
// induced by a sampled node set (the last step of the samplers of Section 4,
// Algorithms 2 and 3; Algorithm 1's adjacency matrix of G_s), with a self
// loop on every node and the normalisation of Eq. "graphsage forward"
// (D^-1 A, D counting the stored entries) or the symmetric one of the GCN
// layer, plus the row gather of the features and labels of V_s (Algorithm
// 1's feature and label lookup).  The full graph stays resident in HBM; only
// the node list of each subgraph arrives from the host.
//
// Entry space.  Before selection, row i of the result is the full row of
// v = nodes[i] with v itself merged in at its sorted position p_i (the
// number of neighbours below v): deg(v) + 1 slots.  The slots of all rows
// are laid end to end (row offsets off[i], an exclusive scan of deg + 1).
// A slot is kept if it is the self loop or a neighbour w != v of V_s
// (map[w] >= 0, map = full id -> position in V_s).  One exclusive scan of
// the keep flags over the whole entry space gives every kept slot its
// output position, and the count before row i's first slot is indptr_s[i].
// Rows come out sorted because V_s is sorted and the map keeps that order.
// Work is split into equal slot chunks over a fixed grid, so a hub row of
// the full graph is shared by many workgroups.
#include <cmath>

#include "abi.hpp"

using namespace gnnprop;

namespace {

constexpr int SCAN_THREADS = 256;
constexpr int SCAN_ITEMS = 8;
constexpr int SCAN_TILE = SCAN_THREADS * SCAN_ITEMS;  // 2048
constexpr int CHUNK_BLOCKS = 1024;  // fixed grid over the entry space
constexpr int ST_RANGE = 1, ST_ORDER = 2, ST_CAPACITY = 4;

// Exclusive scan over a block of 256 threads, each holding SCAN_ITEMS
// consecutive items (blocked arrangement).  lds: 4 int64.
__device__ inline void block_scan(int64_t (&v)[SCAN_ITEMS], int64_t* lds,
                                  int64_t& total) {
  int64_t s = 0;
#pragma unroll
  for (int k = 0; k < SCAN_ITEMS; ++k) {
    const int64_t x = v[k];
    v[k] = s;
    s += x;
  }
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  int64_t inc = s;
#pragma unroll
  for (int d = 1; d < 64; d <<= 1) {
    const int64_t y = __shfl_up(inc, d, 64);
    if (lane >= d) inc += y;
  }
  if (lane == 63) lds[w] = inc;
  __syncthreads();
  int64_t before = 0, tot = 0;
#pragma unroll
  for (int k = 0; k < SCAN_THREADS / 64; ++k) {
    if (k < w) before += lds[k];
    tot += lds[k];
  }
  __syncthreads();
  const int64_t excl = before + inc - s;
#pragma unroll
  for (int k = 0; k < SCAN_ITEMS; ++k) v[k] += excl;
  total = tot;
}

template <typename T>
__device__ inline void load_tile(int64_t N, const T* __restrict__ in, int64_t base,
                                 int64_t (&v)[SCAN_ITEMS]) {
#pragma unroll
  for (int k = 0; k < SCAN_ITEMS; ++k) {
    const int64_t i = base + (int64_t)threadIdx.x * SCAN_ITEMS + k;
    v[k] = i < N ? (int64_t)in[i] : 0;
  }
}

// sums[b] = sum of tile b of in[0..N)
template <typename T>
__global__ __launch_bounds__(SCAN_THREADS) void scan_reduce_kernel(
    int64_t N, const T* __restrict__ in, int64_t* __restrict__ sums) {
  __shared__ int64_t lds[4];
  int64_t v[SCAN_ITEMS];
  load_tile(N, in, (int64_t)blockIdx.x * SCAN_TILE, v);
  int64_t total;
  block_scan(v, lds, total);
  if (threadIdx.x == 0) sums[blockIdx.x] = total;
}

// One block: offs = exclusive scan of sums[0..T), *total = their sum.
__global__ __launch_bounds__(SCAN_THREADS) void scan_top_kernel(
    int64_t T, const int64_t* __restrict__ sums, int64_t* __restrict__ offs,
    int64_t* __restrict__ total) {
  __shared__ int64_t lds[4];
  int64_t carry = 0;
  for (int64_t base = 0; base < T; base += SCAN_TILE) {
    int64_t v[SCAN_ITEMS];
    load_tile(T, sums, base, v);
    int64_t t;
    block_scan(v, lds, t);
#pragma unroll
    for (int k = 0; k < SCAN_ITEMS; ++k) {
      const int64_t i = base + (int64_t)threadIdx.x * SCAN_ITEMS + k;
      if (i < T) offs[i] = carry + v[k];
    }
    carry += t;
  }
  if (threadIdx.x == 0) *total = carry;
}

// out[i] = offs[tile] + exclusive scan within the tile; with offs == NULL
// (a single tile) the block also writes the total to out[N].
template <typename T>
__global__ __launch_bounds__(SCAN_THREADS) void scan_down_kernel(
    int64_t N, const T* __restrict__ in, const int64_t* __restrict__ offs,
    int64_t* __restrict__ out) {
  __shared__ int64_t lds[4];
  int64_t v[SCAN_ITEMS];
  const int64_t base = (int64_t)blockIdx.x * SCAN_TILE;
  load_tile(N, in, base, v);
  int64_t total;
  block_scan(v, lds, total);
  const int64_t o = offs ? offs[blockIdx.x] : 0;
#pragma unroll
  for (int k = 0; k < SCAN_ITEMS; ++k) {
    const int64_t i = base + (int64_t)threadIdx.x * SCAN_ITEMS + k;
    if (i < N) out[i] = o + v[k];
  }
  if (!offs && threadIdx.x == 0) out[N] = total;
}

// out[0..N] = exclusive scan of in[0..N) followed by the total.
// tmp: 2 * ceil(N / SCAN_TILE) int64.
template <typename T>
hipError_t scan_exclusive(int64_t N, const T* in, int64_t* out, int64_t* tmp,
                          hipStream_t s) {
  const int64_t tiles = std::max<int64_t>(1, ceil_div(N, SCAN_TILE));
  if (tiles == 1) {
    scan_down_kernel<T><<<1, SCAN_THREADS, 0, s>>>(N, in, nullptr, out);
    return hipGetLastError();
  }
  int64_t* sums = tmp;
  int64_t* offs = tmp + tiles;
  scan_reduce_kernel<T><<<(unsigned)tiles, SCAN_THREADS, 0, s>>>(N, in, sums);
  scan_top_kernel<<<1, SCAN_THREADS, 0, s>>>(tiles, sums, offs, out + N);
  scan_down_kernel<T><<<(unsigned)tiles, SCAN_THREADS, 0, s>>>(N, in, offs, out);
  return hipGetLastError();
}

// Clears the status word and the count outputs (a kernel, not a memset, so
// that the call can be captured in a graph).
__global__ void induce_clear_kernel(int32_t* __restrict__ status,
                                    int64_t* __restrict__ nnz_out,
                                    int32_t* __restrict__ sub_indptr, int32_t n_s) {
  if (threadIdx.x == 0) {
    *status = 0;
    *nnz_out = 0;
    if (n_s == 0) sub_indptr[0] = 0;
  }
}

// Per sampled row: range and order checks, map[v] = i, deg + 1 slots and the
// self loop's slot p_i.  Rows whose node is out of range keep the self loop
// alone and never touch the full graph.
__global__ __launch_bounds__(256) void induce_rows_kernel(
    int64_t n_full, const int64_t* __restrict__ indptr,
    const int32_t* __restrict__ indices, int32_t n_s,
    const int32_t* __restrict__ nodes, int32_t* __restrict__ map,
    int32_t* __restrict__ slots, int32_t* __restrict__ pself,
    int32_t* __restrict__ status) {
  const int32_t i = blockIdx.x * 256 + threadIdx.x;
  if (i >= n_s) return;
  const int32_t v = nodes[i];
  int bad = (v < 0 || (int64_t)v >= n_full) ? ST_RANGE : 0;
  if (i + 1 < n_s && nodes[i + 1] <= v) bad |= ST_ORDER;
  if (bad & ST_RANGE) {
    slots[i] = 1;
    pself[i] = 0;
  } else {
    map[v] = i;
    const int64_t b = indptr[v];
    const int64_t deg = indptr[v + 1] - b;
    int64_t lo = 0, hi = deg;
    while (lo < hi) {
      const int64_t mid = (lo + hi) >> 1;
      if (indices[b + mid] < v) lo = mid + 1;
      else hi = mid;
    }
    slots[i] = (int32_t)(deg + 1);
    pself[i] = (int32_t)lo;
  }
  if (bad) atomicOr(status, bad);
}

// Row of slot e: the last row r in [lo, hi] with off[r] <= e.
__device__ inline int32_t row_of(const int64_t* __restrict__ off, int32_t lo,
                                 int32_t hi, int64_t e) {
  while (lo < hi) {
    const int32_t mid = (lo + hi + 1) >> 1;
    if (off[mid] <= e) lo = mid;
    else hi = mid - 1;
  }
  return lo;
}

struct EntryArgs {
  int32_t n_s;
  int64_t n_full;
  const int64_t* indptr;
  const int32_t* indices;
  const int32_t* nodes;
  const int32_t* map;
  const int32_t* pself;
  const int64_t* off;  // n_s + 1
};

// Column (position in V_s) that slot k of row i keeps, or -1.
__device__ inline int32_t slot_target(const EntryArgs& a, int32_t i, int64_t k) {
  const int32_t p = a.pself[i];
  if (k == p) return i;
  const int32_t v = a.nodes[i];
  const int32_t w = a.indices[a.indptr[v] + (k - (k > p ? 1 : 0))];
  if (w == v) return -1;  // a loop stored in the full graph counts once
  if (w < 0 || (int64_t)w >= a.n_full) return -1;
  return a.map[w];
}

// The chunk of the entry space this block owns, and its rows.
__device__ inline bool chunk_of(const EntryArgs& a, int64_t& start, int64_t& end,
                                int32_t& r_lo, int32_t& r_hi, int32_t* lds) {
  const int64_t E = a.off[a.n_s];
  const int64_t chunk = ceil_div(E, CHUNK_BLOCKS);
  start = (int64_t)blockIdx.x * chunk;
  end = std::min(E, start + chunk);
  if (start >= end) return false;
  if (threadIdx.x == 0) {
    lds[0] = row_of(a.off, 0, a.n_s - 1, start);
    lds[1] = row_of(a.off, lds[0], a.n_s - 1, end - 1);
  }
  __syncthreads();
  r_lo = lds[0];
  r_hi = lds[1];
  return true;
}

// The chunk's row offsets off[r_lo .. r_hi + 1], staged in LDS when they
// fit, so that each slot finds its row without global reads.
constexpr int ROW_CACHE = 512;

struct Rows {
  const int64_t* off;  // LDS copy (relative to r_lo) or the global array
  int32_t lo, hi, base;
};

__device__ inline Rows stage_rows(const EntryArgs& a, int32_t r_lo, int32_t r_hi,
                                  int64_t* s_off) {
  const int32_t cnt = r_hi - r_lo + 2;
  if (cnt > ROW_CACHE + 1) return Rows{a.off, r_lo, r_hi, 0};
  for (int32_t k = threadIdx.x; k < cnt; k += 256) s_off[k] = a.off[r_lo + k];
  __syncthreads();
  return Rows{s_off, 0, r_hi - r_lo, r_lo};
}

// (row, slot within the row) of entry e
__device__ inline int32_t row_in(const Rows& R, int64_t e, int64_t& k) {
  const int32_t r = row_of(R.off, R.lo, R.hi, e);
  k = e - R.off[r];
  return r + R.base;
}

__global__ __launch_bounds__(256) void induce_count_kernel(EntryArgs a,
                                                           int64_t* __restrict__ counts) {
  __shared__ int32_t rows[2];
  __shared__ int32_t wsum[4];
  __shared__ int64_t s_off[ROW_CACHE + 1];
  int64_t start, end;
  int32_t r_lo, r_hi;
  if (!chunk_of(a, start, end, r_lo, r_hi, rows)) {
    if (threadIdx.x == 0) counts[blockIdx.x] = 0;
    return;
  }
  const Rows R = stage_rows(a, r_lo, r_hi, s_off);
  int32_t c = 0;
  for (int64_t e = start + threadIdx.x; e < end; e += 256) {
    int64_t k;
    const int32_t i = row_in(R, e, k);
    c += slot_target(a, i, k) >= 0;
  }
#pragma unroll
  for (int d = 32; d > 0; d >>= 1) c += __shfl_xor(c, d, 64);
  if ((threadIdx.x & 63) == 0) wsum[threadIdx.x >> 6] = c;
  __syncthreads();
  if (threadIdx.x == 0) counts[blockIdx.x] = (int64_t)wsum[0] + wsum[1] + wsum[2] + wsum[3];
}

// Writes the kept slots at their scanned positions and indptr_s; block 0
// also writes the total and checks it against the capacity.
__global__ __launch_bounds__(256) void induce_fill_kernel(
    EntryArgs a, const int64_t* __restrict__ boff, int64_t capacity,
    int32_t* __restrict__ sub_indptr, int32_t* __restrict__ sub_indices,
    int64_t* __restrict__ nnz_out, int32_t* __restrict__ status) {
  __shared__ int32_t rows[2];
  __shared__ int32_t wcnt[4];
  __shared__ int64_t s_off[ROW_CACHE + 1];
  if (blockIdx.x == 0 && threadIdx.x == 0) {
    const int64_t total = boff[CHUNK_BLOCKS];
    *nnz_out = total;
    sub_indptr[a.n_s] = (int32_t)std::min<int64_t>(total, INT32_MAX);
    if (total > capacity || total > INT32_MAX) atomicOr(status, ST_CAPACITY);
  }
  int64_t start, end;
  int32_t r_lo, r_hi;
  if (!chunk_of(a, start, end, r_lo, r_hi, rows)) return;
  const Rows R = stage_rows(a, r_lo, r_hi, s_off);
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  int64_t run = boff[blockIdx.x];
  for (int64_t base = start; base < end; base += 256) {
    const int64_t e = base + threadIdx.x;
    int32_t i = 0, t = -1;
    int64_t k = -1;
    if (e < end) {
      i = row_in(R, e, k);
      t = slot_target(a, i, k);
    }
    const uint64_t m = __ballot(t >= 0);
    const int32_t below = __popcll(m & ((1ull << lane) - 1ull));
    if (lane == 0) wcnt[w] = __popcll(m);
    __syncthreads();
    int32_t before = 0;
    for (int k = 0; k < w; ++k) before += wcnt[k];
    const int32_t tile = wcnt[0] + wcnt[1] + wcnt[2] + wcnt[3];
    __syncthreads();
    const int64_t pos = run + before + below;
    if (e < end) {
      if (k == 0) sub_indptr[i] = (int32_t)std::min<int64_t>(pos, INT32_MAX);
      if (t >= 0 && pos < capacity) sub_indices[pos] = t;
    }
    run += tile;
  }
}

// Values of row i (one wavefront per row) and the map entry reset.
__global__ __launch_bounds__(256) void induce_values_kernel(
    int32_t n_s, int64_t n_full, const int32_t* __restrict__ nodes,
    int32_t* __restrict__ map, const int32_t* __restrict__ sub_indptr,
    const int32_t* __restrict__ sub_indices, float* __restrict__ sub_values,
    int64_t capacity, int32_t norm) {
  const int32_t i = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (i >= n_s) return;
  const int64_t b = sub_indptr[i];
  const int64_t e = std::min<int64_t>(sub_indptr[i + 1], capacity);
  const double lu = (double)(sub_indptr[i + 1] - sub_indptr[i]);
  for (int64_t j = b + lane; j < e; j += 64) {
    double val;
    if (norm == GNN_NORM_ROW) {
      val = 1.0 / lu;
    } else {
      const int32_t k = sub_indices[j];
      val = 1.0 / sqrt(lu * (double)(sub_indptr[k + 1] - sub_indptr[k]));
    }
    sub_values[j] = (float)val;
  }
  const int32_t v = nodes[i];
  if (lane == 0 && v >= 0 && (int64_t)v < n_full) map[v] = -1;
}

// dst row r = src row index[r] (width floats); out-of-range ids give zeros.
template <bool VEC>
__global__ __launch_bounds__(256) void gather_rows_kernel(
    int32_t rows, const int32_t* __restrict__ index, int32_t width,
    const float* __restrict__ src, int64_t ld_src, int64_t src_rows,
    float* __restrict__ dst, int64_t ld_dst) {
  const int32_t r = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (r >= rows) return;
  const int32_t s = index[r];
  const bool ok = s >= 0 && (int64_t)s < src_rows;
  const float* in = src + (int64_t)(ok ? s : 0) * ld_src;
  float* out = dst + (int64_t)r * ld_dst;
  if (VEC) {
    const int32_t w4 = width >> 2;
    for (int32_t c = lane; c < w4; c += 64) {
      const float4 x = ok ? reinterpret_cast<const float4*>(in)[c]
                          : make_float4(0.f, 0.f, 0.f, 0.f);
      reinterpret_cast<float4*>(out)[c] = x;
    }
  } else {
    for (int32_t c = lane; c < width; c += 64) out[c] = ok ? in[c] : 0.f;
  }
}

struct InduceLayout {
  size_t off_slots, off_pself, off_off, off_tmp, off_counts, off_boff, total;
};

InduceLayout induce_layout(int32_t n_s) {
  InduceLayout o;
  const int64_t tiles = std::max<int64_t>(1, ceil_div(n_s, SCAN_TILE));
  size_t p = 0;
  o.off_slots = p;
  p += round_up((size_t)std::max(n_s, 1) * 4, 256);
  o.off_pself = p;
  p += round_up((size_t)std::max(n_s, 1) * 4, 256);
  o.off_off = p;
  p += round_up((size_t)(n_s + 1) * 8, 256);
  o.off_tmp = p;
  p += round_up((size_t)tiles * 2 * 8, 256);
  o.off_counts = p;
  p += round_up((size_t)CHUNK_BLOCKS * 8, 256);
  o.off_boff = p;
  p += round_up((size_t)(CHUNK_BLOCKS + 1) * 8, 256);
  o.total = p;
  return o;
}

}  // namespace

extern "C" {

size_t gnn_induce_workspace_bytes(int32_t n_s) {
  if (n_s < 0) return 0;
  return induce_layout(n_s).total;
}

gnn_status gnn_induce_subgraph(int64_t n_full, int64_t nnz_full,
                               const int64_t* indptr, const int32_t* indices,
                               int32_t n_s,
                               const int32_t* nodes, int32_t norm, int32_t* map,
                               int64_t capacity, int32_t* sub_indptr,
                               int32_t* sub_indices, float* sub_values,
                               int64_t* nnz_out, int32_t* status_out,
                               void* workspace, size_t workspace_bytes,
                               hipStream_t stream) {
  if (n_full < 0 || n_full > INT32_MAX || nnz_full < 0 || n_s < 0 || capacity < 0)
    return GNN_ERR_SHAPE;
  if (norm != GNN_NORM_ROW && norm != GNN_NORM_SYM) return GNN_ERR_UNSUPPORTED;
  if (!sub_indptr || !nnz_out || !status_out) return GNN_ERR_NULL;
  if (!buf16(workspace)) return GNN_ERR_UNSUPPORTED;
  if (n_s > 0 && (!indptr || !nodes || !map || !sub_indices || !sub_values || !workspace))
    return GNN_ERR_NULL;
  if (n_s > 0 && nnz_full > 0 && !indices) return GNN_ERR_NULL;
  if (n_s > 0 && capacity < n_s) return GNN_ERR_SHAPE;  // every row keeps its loop
  const InduceLayout o = induce_layout(n_s);
  if (n_s > 0 && workspace_bytes < o.total) return GNN_ERR_WORKSPACE;
  {
    const void* outs[] = {map, sub_indptr, sub_indices, sub_values, nnz_out, status_out,
                          workspace};
    const size_t outb[] = {(size_t)n_full * 4, (size_t)(n_s + 1) * 4,
                           (size_t)capacity * 4, (size_t)capacity * 4, 8, 4,
                           n_s > 0 ? o.total : 0};
    const void* ins[] = {indptr, indices, nodes};
    const size_t inb[] = {(size_t)(n_full + 1) * 8, (size_t)nnz_full * 4,
                          (size_t)n_s * 4};
    for (int k = 0; k < 7; ++k) {
      for (int j = 0; j < 3; ++j)
        if (ranges_overlap(outs[k], outb[k], ins[j], inb[j])) return GNN_ERR_ALIAS;
      for (int j = 0; j < k; ++j)
        if (ranges_overlap(outs[k], outb[k], outs[j], outb[j])) return GNN_ERR_ALIAS;
    }
  }
  timer_begin(GNN_K_INDUCE, stream);
  induce_clear_kernel<<<1, 64, 0, stream>>>(status_out, nnz_out, sub_indptr, n_s);
  if (n_s == 0) {  // empty node set: indptr_s = {0}, nnz 0, status 0
    timer_end(GNN_K_INDUCE, 0.0, stream);
    GNN_HIP(hipGetLastError());
    return GNN_OK;
  }
  char* ws = static_cast<char*>(workspace);
  int32_t* slots = reinterpret_cast<int32_t*>(ws + o.off_slots);
  int32_t* pself = reinterpret_cast<int32_t*>(ws + o.off_pself);
  int64_t* off = reinterpret_cast<int64_t*>(ws + o.off_off);
  int64_t* tmp = reinterpret_cast<int64_t*>(ws + o.off_tmp);
  int64_t* counts = reinterpret_cast<int64_t*>(ws + o.off_counts);
  int64_t* boff = reinterpret_cast<int64_t*>(ws + o.off_boff);
  induce_rows_kernel<<<(unsigned)ceil_div(n_s, 256), 256, 0, stream>>>(
      n_full, indptr, indices, n_s, nodes, map, slots, pself, status_out);
  GNN_HIP(hipGetLastError());
  GNN_HIP(scan_exclusive<int32_t>(n_s, slots, off, tmp, stream));
  EntryArgs a{n_s, n_full, indptr, indices, nodes, map, pself, off};
  induce_count_kernel<<<CHUNK_BLOCKS, 256, 0, stream>>>(a, counts);
  GNN_HIP(hipGetLastError());
  GNN_HIP(scan_exclusive<int64_t>(CHUNK_BLOCKS, counts, boff, tmp, stream));
  induce_fill_kernel<<<CHUNK_BLOCKS, 256, 0, stream>>>(a, boff, capacity, sub_indptr,
                                                       sub_indices, nnz_out, status_out);
  GNN_HIP(hipGetLastError());
  induce_values_kernel<<<(unsigned)ceil_div(n_s, 4), 256, 0, stream>>>(
      n_s, n_full, nodes, map, sub_indptr, sub_indices, sub_values, capacity, norm);
  timer_end(GNN_K_INDUCE, 0.0, stream);
  GNN_HIP(hipGetLastError());
  return GNN_OK;
}

gnn_status gnn_gather_rows(int32_t rows, const int32_t* index, int32_t width,
                           const float* src, int64_t ld_src, int64_t src_rows,
                           float* dst, int64_t ld_dst, hipStream_t stream) {
  if (rows < 0 || width < 0 || src_rows < 0) return GNN_ERR_SHAPE;
  if (rows == 0 || width == 0) return GNN_OK;
  if (!index || !dst || (src_rows > 0 && !src)) return GNN_ERR_NULL;
  if (ld_src < width || ld_dst < width) return GNN_ERR_SHAPE;
  if (ranges_overlap(dst, mat_bytes(rows, width, ld_dst), src, mat_bytes(src_rows, width, ld_src)) ||
      ranges_overlap(dst, mat_bytes(rows, width, ld_dst), index, (size_t)rows * 4))
    return GNN_ERR_ALIAS;
  const bool vec = width % 4 == 0 && ld_src % 4 == 0 && ld_dst % 4 == 0 &&
                   reinterpret_cast<uintptr_t>(src) % 16 == 0 &&
                   reinterpret_cast<uintptr_t>(dst) % 16 == 0;
  timer_begin(GNN_K_GATHER, stream);
  if (vec)
    gather_rows_kernel<true><<<(unsigned)ceil_div(rows, 4), 256, 0, stream>>>(
        rows, index, width, src, ld_src, src_rows, dst, ld_dst);
  else
    gather_rows_kernel<false><<<(unsigned)ceil_div(rows, 4), 256, 0, stream>>>(
        rows, index, width, src, ld_src, src_rows, dst, ld_dst);
  timer_end(GNN_K_GATHER, 8.0 * rows * width, stream);
  GNN_HIP(hipGetLastError());
  return GNN_OK;
}

}  // extern "C"
