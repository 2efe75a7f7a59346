// Argument checks and launch helpers shared by the C-ABI translation units.
#pragma once

#include <cstring>

#include "internal.hpp"

namespace gnnprop {

#define GNN_HIP(expr)                         \
  do {                                        \
    if ((expr) != hipSuccess) return GNN_ERR_HIP; \
  } while (0)

inline bool ranges_overlap(const void* a, size_t an, const void* b, size_t bn) {
  if (!a || !b || an == 0 || bn == 0) return false;
  const char* pa = static_cast<const char*>(a);
  const char* pb = static_cast<const char*>(b);
  return pa < pb + bn && pb < pa + an;
}

// Workspace, saved and plan buffers: the kernels access them 16 bytes at a
// time (NULL passes; whether one is required is checked separately).
inline bool buf16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

inline size_t mat_bytes(int64_t rows, int64_t cols, int64_t ld) {
  if (rows <= 0 || cols <= 0) return 0;
  return (size_t)(((rows - 1) * ld + cols) * 4);
}

inline gnn_status check_csr(const gnn_csr* c, bool need_vals, bool need_vals_t) {
  if (!c) return GNN_ERR_NULL;
  if (c->n < 0 || c->nnz < 0 || c->nnz > INT32_MAX) return GNN_ERR_SHAPE;
  if (!c->indptr) return GNN_ERR_NULL;
  if (c->nnz > 0 && !c->indices) return GNN_ERR_NULL;
  if (need_vals && c->nnz > 0 && !c->values) return GNN_ERR_NULL;
  if (need_vals_t && c->nnz > 0 && !c->values_t) return GNN_ERR_NULL;
  if (!buf16(c->plan)) return GNN_ERR_UNSUPPORTED;
  return GNN_OK;
}

// rownorm: A_s = D^-1 A taken from the pattern alone (GNN_FLAG_ROW_NORMALIZED);
// the value arrays are then not read.
inline SpmmCall spmm_call(const gnn_csr* c, bool transpose, int32_t w,
                   const float* in, int64_t ld_in, float* out, int64_t ld_out,
                   bool rownorm = false) {
  SpmmCall s;
  memset(&s, 0, sizeof(s));
  s.n = c->n;
  s.nnz = c->nnz;
  s.indptr = c->indptr;
  s.indices = c->indices;
  s.vals = rownorm ? nullptr : transpose ? c->values_t : c->values;
  s.weights = !rownorm ? SPMM_W_VALUES : transpose ? SPMM_W_COL_DEG : SPMM_W_ROW_SCALE;
  s.plan = c->plan;
  s.w = w;
  s.in = in;
  s.ld_in = ld_in;
  s.out = out;
  s.ld_out = ld_out;
  s.epilogue = SPMM_STORE;
  return s;
}

}  // namespace gnnprop
