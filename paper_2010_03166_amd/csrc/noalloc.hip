// gnn_csr_validate_noalloc: the CSR check of gnn_csr_validate for callers
// that cannot allocate device memory.  gnn_csr_validate allocates (and
// frees) the one status word its kernel writes; here that word lives in a
// file-scope device array, `scratch`, which every call on a device shares.
//
// Host code never passes `scratch` itself to a kernel or a copy: in host code
// the name stands for a host-side shadow, not for device memory.  The device
// address of each device's copy comes from hipGetSymbolAddress, taken once
// per device with that device current, and is what the kernels receive.
#include <mutex>

#include "abi.hpp"

namespace gnnprop {
namespace {

// 256 bytes per device, held until the process ends.  The check uses word 0
// (the status word), whatever the size of the graph.
constexpr int SCRATCH_WORDS = 64;
__device__ __align__(256) int32_t scratch[SCRATCH_WORDS];

constexpr int MAX_DEVICES = 64;
std::mutex g_scratch_mu;
int32_t* g_scratch_ptr[MAX_DEVICES];  // device address of `scratch`, per device

__global__ __launch_bounds__(64) void clear_words_kernel(int32_t* __restrict__ p,
                                                         int32_t count) {
  const int i = threadIdx.x;
  if (i < count) p[i] = 0;
}

// The device address of the current device's `scratch` (looked up on the
// first call on that device).
gnn_status scratch_ptr(int32_t** out) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0) return GNN_ERR_HIP;
  if (dev >= MAX_DEVICES) return GNN_ERR_UNSUPPORTED;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p)
      return GNN_ERR_HIP;
    g_scratch_ptr[dev] = static_cast<int32_t*>(p);
  }
  *out = g_scratch_ptr[dev];
  return GNN_OK;
}

}  // namespace
}  // namespace gnnprop

using namespace gnnprop;

extern "C" gnn_status gnn_csr_validate_noalloc(const gnn_csr* csr,
                                               int32_t require_symmetric,
                                               hipStream_t stream) {
  gnn_status st = check_csr(csr, false, false);
  if (st != GNN_OK) return st;
  int32_t* bad = nullptr;
  if ((st = scratch_ptr(&bad)) != GNN_OK) return st;
  // the array still holds the last call's status: clear it first
  clear_words_kernel<<<1, 64, 0, stream>>>(bad, 1);
  hipError_t e = hipGetLastError();
  if (e == hipSuccess)
    e = validate_csr(csr->n, csr->nnz, csr->indptr, csr->indices,
                     require_symmetric, bad, stream);
  int32_t h_bad = 0;
  if (e == hipSuccess)
    e = hipMemcpyAsync(&h_bad, bad, sizeof(int32_t), hipMemcpyDeviceToHost,
                       stream);
  if (e == hipSuccess) e = hipStreamSynchronize(stream);
  if (e != hipSuccess) return GNN_ERR_HIP;
  return h_bad ? GNN_ERR_CSR : GNN_OK;
}
