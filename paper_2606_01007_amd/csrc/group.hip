// Grouping objective of Sec. 3.3 (eq. grouping-objective) for many placements: the within-group
// affinity  obj[p][l] = sum_m sum_{e != e' on GPU m} A-tilde_l(e, e'),  accumulated in float64.
//
// One workgroup per (placement, layer); consecutive workgroups share the layer, so the layer's
// A-tilde rows stay in L2 while the placements of that layer are scored.  Thread e reads the GPU of
// every expert from LDS (broadcast reads) and adds the entries of its own A-tilde row whose column
// sits on the same GPU: about C_m - 1 gathered floats per expert.
#include "tacg_internal.h"

namespace tacg {
namespace {

constexpr int kThreads = 256;

__global__ __launch_bounds__(kThreads) void group_objective_kernel(const float* __restrict__ a_tilde, int L, int E,
                                                                   const uint8_t* __restrict__ primary, int G,
                                                                   double* __restrict__ obj, uint32_t* d_err) {
  __shared__ uint8_t gpu[TACG_MAX_EXPERTS];
  __shared__ double part[kThreads / 64];
  const int p = blockIdx.x, l = blockIdx.y;
  const int e = threadIdx.x;
  uint32_t err = 0;
  if (e < E) {
    uint8_t g = primary[(static_cast<int64_t>(p) * L + l) * E + e];
    if (g >= G) {
      err = TACG_ERR_TABLE;
      g = 0xFF;  // left out of every group
    }
    gpu[e] = g;
  }
  __syncthreads();
  double acc = 0.0;
  if (e < E && gpu[e] != 0xFF) {
    const uint8_t ge = gpu[e];
    const float* row = a_tilde + (static_cast<int64_t>(l) * E + e) * E;
    for (int e2 = 0; e2 < E; ++e2)
      if (e2 != e && gpu[e2] == ge) acc += static_cast<double>(row[e2]);
  }
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) acc += __shfl_xor(acc, o, 64);
  if ((threadIdx.x & 63) == 0) part[threadIdx.x >> 6] = acc;
  __syncthreads();
  if (threadIdx.x == 0) {
    double s = 0.0;
    for (int w = 0; w < kThreads / 64; ++w) s += part[w];
    obj[static_cast<int64_t>(p) * L + l] = s;
  }
  if (err) atomicOr(d_err, err);
}

}  // namespace

int launch_group_objective(const float* a_tilde, int32_t L, int32_t E, const uint8_t* primary, int32_t P, int32_t G,
                           double* obj, uint32_t* d_err, hipStream_t stream) {
  hipLaunchKernelGGL(group_objective_kernel, dim3(P, L), dim3(kThreads), 0, stream, a_tilde, L, E, primary, G, obj,
                     d_err);
  return hipGetLastError() == hipSuccess ? TACG_OK : TACG_E_DEVICE;
}

}  // namespace tacg
