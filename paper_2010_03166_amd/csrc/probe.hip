// Measurement aid, not part of the method: the sustained rate of the matrix
// cores on the running device, and the shader clock they run at under that
// load.  Every wavefront issues a fixed number of register-operand MFMAs on
// four independent accumulators (no memory traffic in the loop), at the
// occupancy of the split-product GEMM (512-thread workgroups, two per CU).
// The first wavefront of workgroup 0 reads the shader-clock counter
// (s_memtime) and the 100 MHz real-time counter (s_memrealtime) around its
// loop; their ratio gives the clock.  The caller times the launch.
#include "abi.hpp"

namespace gnnprop {

namespace {

typedef float probe_f32x16 __attribute__((ext_vector_type(16)));
typedef __bf16 probe_bf16x8 __attribute__((ext_vector_type(8)));

template <int KIND>
__global__ __launch_bounds__(512) void mfma_probe_kernel(int32_t iters, float* __restrict__ sink,
                                                         uint64_t* __restrict__ clocks) {
  const int tid = threadIdx.x;
  probe_f32x16 acc[4];
#pragma unroll
  for (int u = 0; u < 4; ++u)
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[u][r] = 0.f;
  const bool timer = blockIdx.x == 0 && tid == 0;
  uint64_t t0 = 0, r0 = 0;
  if (timer) {
    t0 = __builtin_amdgcn_s_memtime();
    r0 = __builtin_amdgcn_s_memrealtime();
  }
  if (KIND == GNN_PROBE_MFMA_BF16) {
    probe_bf16x8 a, b;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      a[i] = (__bf16)(1e-3f * (float)(tid + i));
      b[i] = (__bf16)(1e-3f * (float)(tid - i));
    }
    for (int it = 0; it < iters; ++it)
#pragma unroll
      for (int u = 0; u < 4; ++u)
        acc[u] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, acc[u], 0, 0, 0);
  } else {
    const float a = 1e-3f * (float)tid, b = 2e-3f * (float)tid;
    for (int it = 0; it < iters; ++it)
#pragma unroll
      for (int u = 0; u < 4; ++u)
        acc[u] = __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, acc[u], 0, 0, 0);
  }
  if (timer) {
    const uint64_t t1 = __builtin_amdgcn_s_memtime();
    const uint64_t r1 = __builtin_amdgcn_s_memrealtime();
    clocks[0] = t1 - t0;
    clocks[1] = r1 - r0;
  }
  // the sums keep the products live
  float s = 0.f;
#pragma unroll
  for (int u = 0; u < 4; ++u)
#pragma unroll
    for (int r = 0; r < 16; ++r) s += acc[u][r];
  sink[(int64_t)blockIdx.x * 512 + tid] = s;
}

}  // namespace

}  // namespace gnnprop

using namespace gnnprop;

extern "C" gnn_status gnn_mfma_rate_probe(int32_t kind, int32_t blocks, int32_t iters,
                                          float* sink, uint64_t* clocks, hipStream_t stream) {
  if (kind != GNN_PROBE_MFMA_BF16 && kind != GNN_PROBE_MFMA_F32) return GNN_ERR_UNSUPPORTED;
  if (blocks < 1 || blocks > GNN_PROBE_MAX_BLOCKS || iters < 1 || iters > GNN_PROBE_MAX_ITERS)
    return GNN_ERR_SHAPE;
  if (!sink || !clocks) return GNN_ERR_NULL;
  if (reinterpret_cast<uintptr_t>(sink) % 4 != 0 || reinterpret_cast<uintptr_t>(clocks) % 8 != 0)
    return GNN_ERR_UNSUPPORTED;
  if (ranges_overlap(sink, (size_t)blocks * 512 * sizeof(float), clocks, 2 * sizeof(uint64_t)))
    return GNN_ERR_ALIAS;
  if (kind == GNN_PROBE_MFMA_BF16)
    mfma_probe_kernel<GNN_PROBE_MFMA_BF16><<<blocks, 512, 0, stream>>>(iters, sink, clocks);
  else
    mfma_probe_kernel<GNN_PROBE_MFMA_F32><<<blocks, 512, 0, stream>>>(iters, sink, clocks);
  GNN_HIP(hipGetLastError());
  return GNN_OK;
}
