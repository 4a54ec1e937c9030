// Grouping objective of Sec. 3.3 (eq. grouping-objective) for many placements: the within-group
// affinity  obj[p][l] = sum_m sum_{e != e' on GPU m} A-tilde_l(e, e'),  accumulated in float64.
//
// One workgroup per (placement, layer); consecutive workgroups share the layer, so the layer's
// A-tilde rows stay in L2 while the placements of that layer are scored.  The workgroup first lists
// the experts of every GPU in increasing id order (per-wave ballots give each expert its rank in its
// GPU's list), then thread e adds the entries of its own A-tilde row at the other members of its GPU:
// about C_m - 1 gathered floats and as many loop steps per expert, in increasing column order.
#include "tacg_internal.h"

namespace tacg {
namespace {

constexpr int kThreads = 256;

__global__ __launch_bounds__(kThreads) void group_objective_kernel(const float* __restrict__ a_tilde, int L, int E,
                                                                   const uint8_t* __restrict__ primary, int G,
                                                                   double* __restrict__ obj, uint32_t* d_err) {
  constexpr int kWaves = kThreads / 64;
  __shared__ unsigned long long lanes_of[kWaves][TACG_MAX_GPUS];  // lanes of each wave holding GPU m
  __shared__ int start[TACG_MAX_GPUS + 1];                        // list offsets per GPU
  __shared__ uint8_t member[TACG_MAX_EXPERTS];                    // experts grouped by GPU, ids increasing
  __shared__ double part[kWaves];
  const int p = blockIdx.x, l = blockIdx.y;
  const int e = threadIdx.x;
  const int lane = e & 63, wave = e >> 6;
  uint32_t err = 0;
  uint32_t g = 0xFF;  // 0xFF: no expert, or left out of every group (a table error)
  if (e < E) {
    g = primary[(static_cast<int64_t>(p) * L + l) * E + e];
    if (g >= static_cast<uint32_t>(G)) {
      err = TACG_ERR_TABLE;
      g = 0xFF;
    }
  }
  for (int m = 0; m < G; ++m) {
    const unsigned long long b = __ballot(g == static_cast<uint32_t>(m));
    if (lane == 0) lanes_of[wave][m] = b;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    int s = 0;
    for (int m = 0; m < G; ++m) {
      start[m] = s;
      for (int w = 0; w < kWaves; ++w) s += __popcll(lanes_of[w][m]);
    }
    start[G] = s;
  }
  __syncthreads();
  if (g != 0xFF) {
    int rank = __popcll(lanes_of[wave][g] & ((1ull << lane) - 1ull));
    for (int w = 0; w < wave; ++w) rank += __popcll(lanes_of[w][g]);
    member[start[g] + rank] = static_cast<uint8_t>(e);
  }
  __syncthreads();
  double acc = 0.0;
  if (g != 0xFF) {
    const float* row = a_tilde + (static_cast<int64_t>(l) * E + e) * E;
    const int b0 = start[g], b1 = start[g + 1];
#pragma unroll 4
    for (int i = b0; i < b1; ++i) {
      const int e2 = member[i];
      if (e2 != e) acc += static_cast<double>(row[e2]);
    }
  }
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) acc += __shfl_xor(acc, o, 64);
  if (lane == 0) part[wave] = acc;
  __syncthreads();
  if (threadIdx.x == 0) {
    double s = 0.0;
    for (int w = 0; w < kWaves; ++w) s += part[w];
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
