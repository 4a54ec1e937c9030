// Family preferences and the task-modulated co-activation graph (Sec. 3.3, eqs.
// usage-coact-advantage, coact-advantage, zscore, soft-score, family-pref, same-family-kernel,
// task-modulated-graph).  Internal arithmetic is float64; outputs are float32.
//
// Four passes per call (all small next to the trace passes; C is read once):
//   rw_nf     grid (L, F), one wave each: N_f = sum_i D_f[i] / k of every (layer, family).
//   rw_rows   grid (L, row blocks): per row i and family f the co-activation strength
//             c_f(i) = sum_{j != i} C_f[i][j] / N_f, the pooled A-bar[i][j] = mean_f C_f[i][j] / N_f
//             (zero diagonal) and the layer maximum of A-bar (atomic max on the float64 bit pattern,
//             valid because every value is >= 0).  A wave reads the row of eight families at once.
//   rw_z      grid (L, F), one thread per expert: usage u_f = D_f / (N_f k), advantages against the
//             mean of the other families, z-scores over experts (population std), s = z(du) + z(dc).
//   rw_graph  grid (L, row blocks): the softmax over f of the layer's scores into LDS (the first row
//             block also writes the preferences), then A-hat = A-bar / max, A_task = P P^T, A-tilde.
#include "tacg_internal.h"

namespace tacg {
namespace {

constexpr int kRows = 16;  // rows of a layer per workgroup in rw_rows / rw_graph

struct RwWs {
  double* c;          // [L][F][E]
  double* abar;       // [L][E][E]
  uint64_t* maxbits;  // [L]
  double* s;          // [L][F][E]  soft scores divided by tau
  double* nf;         // [L][F]     tokens per family
};

RwWs carve_rw(void* ws, int32_t F, int32_t L, int32_t E, size_t* used = nullptr) {
  Carver c{static_cast<char*>(ws), 0};
  RwWs r;
  r.c = c.take<double>(static_cast<size_t>(L) * F * E);
  r.abar = c.take<double>(static_cast<size_t>(L) * E * E);
  r.maxbits = c.take<uint64_t>(static_cast<size_t>(L));
  r.s = c.take<double>(static_cast<size_t>(L) * F * E);
  r.nf = c.take<double>(static_cast<size_t>(L) * F);
  if (used) *used = c.used;
  return r;
}

__device__ __forceinline__ double wave_sum(double v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

__device__ __forceinline__ double wave_max(double v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v = fmax(v, __shfl_xor(v, o, 64));
  return v;
}

// Sum over the workgroup (blockDim.x a multiple of 64, <= 1024); every thread gets the result.
__device__ double block_sum(double v, double* red) {
  v = wave_sum(v);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, nw = blockDim.x >> 6;
  __syncthreads();
  if (lane == 0) red[wave] = v;
  __syncthreads();
  double t = 0.0;
  for (int i = 0; i < nw; ++i) t += red[i];
  return t;
}

// N_f of every (layer, family): one wave per pair, lanes over experts (an exact integer sum); the
// (l, 0) wave also clears the layer's maximum.
__global__ __launch_bounds__(64) void rw_nf(const uint32_t* __restrict__ D, int F, int L, int E, int k, RwWs ws) {
  const int l = blockIdx.x, f = blockIdx.y, lane = threadIdx.x;
  const uint32_t* d = D + (static_cast<int64_t>(f) * L + l) * E;
  unsigned long long s = 0;
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int e = lane + 64 * q;
    if (e < E) s += d[e];
  }
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) s += __shfl_xor(s, o, 64);
  if (lane == 0) {
    ws.nf[static_cast<int64_t>(l) * F + f] = static_cast<double>(s) / k;
    if (f == 0) ws.maxbits[l] = 0;
  }
}

constexpr int kFamChunk = 8;  // family rows of C read together in rw_rows

__global__ __launch_bounds__(256) void rw_rows(const uint32_t* __restrict__ C, int F, int L, int E, RwWs ws) {
  __shared__ double inv_n[TACG_MAX_FAMILIES];
  const int l = blockIdx.x;
  for (int f = threadIdx.x; f < F; f += blockDim.x) {
    const double n = ws.nf[static_cast<int64_t>(l) * F + f];
    inv_n[f] = n > 0 ? 1.0 / n : 0.0;
  }
  __syncthreads();
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, nw = blockDim.x >> 6;
  const int r0 = blockIdx.y * kRows, r1 = min(E, r0 + kRows);
  double mx = 0.0;
  for (int i = r0 + wave; i < r1; i += nw) {
    double ab[4] = {0, 0, 0, 0};
    for (int f0 = 0; f0 < F; f0 += kFamChunk) {
      // the row of up to eight families in flight (family index clamped into range)
      uint32_t v[kFamChunk][4];
#pragma unroll
      for (int u = 0; u < kFamChunk; ++u) {
        const int f = min(f0 + u, F - 1);
        const uint32_t* row = C + ((static_cast<int64_t>(f) * L + l) * E + i) * E;
#pragma unroll
        for (int q = 0; q < 4; ++q) v[u][q] = row[min(lane + 64 * q, E - 1)];
      }
#pragma unroll
      for (int u = 0; u < kFamChunk; ++u) {
        const int f = f0 + u;
        if (f >= F) break;
        double rs = 0.0;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int j = lane + 64 * q;
          if (j < E && j != i) {
            const double a = v[u][q] * inv_n[f];
            rs += a;
            ab[q] += a;
          }
        }
        rs = wave_sum(rs);
        if (lane == 0) ws.c[(static_cast<int64_t>(l) * F + f) * E + i] = rs;
      }
    }
    double* arow = ws.abar + (static_cast<int64_t>(l) * E + i) * E;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int j = lane + 64 * q;
      if (j < E) {
        const double v = ab[q] / F;
        arow[j] = v;
        mx = fmax(mx, v);
      }
    }
  }
  mx = wave_max(mx);
  if (lane == 0 && mx > 0.0) atomicMax(reinterpret_cast<unsigned long long*>(ws.maxbits + l),
                                       static_cast<unsigned long long>(__double_as_longlong(mx)));
}

// One workgroup per (layer, family), one thread per expert (E <= 256 = blockDim): the family's
// soft score s / tau of every expert.
__global__ __launch_bounds__(256) void rw_z(const uint32_t* __restrict__ D, int F, int L, int E, int k,
                                            double tau, double eps, RwWs ws) {
  __shared__ double red[16];
  const int l = blockIdx.x, f = blockIdx.y;
  const int e = threadIdx.x;
  const bool on = e < E;
  const double* nf = ws.nf + static_cast<int64_t>(l) * F;
  double du = 0.0, dc = 0.0;
  if (on) {
    // sums over families of u and c for this expert, in family order
    double su = 0.0, sc = 0.0, uf = 0.0, cf = 0.0;
    for (int g = 0; g < F; ++g) {
      const double n = nf[g];
      const double u = n > 0 ? D[(static_cast<int64_t>(g) * L + l) * E + e] / (n * k) : 0.0;
      const double c = ws.c[(static_cast<int64_t>(l) * F + g) * E + e];
      su += u;
      sc += c;
      if (g == f) {
        uf = u;
        cf = c;
      }
    }
    du = uf - (su - uf) / (F - 1);
    dc = cf - (sc - cf) / (F - 1);
  }
  const double mu_u = block_sum(on ? du : 0.0, red) / E;
  const double mu_c = block_sum(on ? dc : 0.0, red) / E;
  const double vu = block_sum(on ? (du - mu_u) * (du - mu_u) : 0.0, red) / E;
  const double vc = block_sum(on ? (dc - mu_c) * (dc - mu_c) : 0.0, red) / E;
  if (on) {
    const double z = (du - mu_u) / (sqrt(vu) + eps) + (dc - mu_c) / (sqrt(vc) + eps);
    ws.s[(static_cast<int64_t>(l) * F + f) * E + e] = z / tau;
  }
}

__global__ __launch_bounds__(256) void rw_graph(int F, int L, int E, double alpha, float* __restrict__ pref,
                                                float* __restrict__ a_tilde, float* __restrict__ a_hat, RwWs ws) {
  extern __shared__ double P[];  // [F][E] preferences of the layer
  const int l = blockIdx.x;
  // softmax over families of the scores, one thread per expert
  {
    const int e = threadIdx.x;
    if (e < E) {
      const double* sl = ws.s + static_cast<int64_t>(l) * F * E;
      double zmax = -INFINITY;
      for (int f = 0; f < F; ++f) zmax = fmax(zmax, sl[f * E + e]);
      double den = 0.0;
      for (int f = 0; f < F; ++f) den += exp(sl[f * E + e] - zmax);
      for (int f = 0; f < F; ++f) {
        const double p = exp(sl[f * E + e] - zmax) / den;
        P[f * E + e] = p;
        if (blockIdx.y == 0) pref[(static_cast<int64_t>(l) * E + e) * F + f] = static_cast<float>(p);
      }
    }
  }
  __syncthreads();
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, nw = blockDim.x >> 6;
  const double mx = __longlong_as_double(static_cast<long long>(ws.maxbits[l]));
  const double inv = mx > 0.0 ? 1.0 / mx : 0.0;
  const int r0 = blockIdx.y * kRows, r1 = min(E, r0 + kRows);
  for (int i = r0 + wave; i < r1; i += nw) {
    const double* arow = ws.abar + (static_cast<int64_t>(l) * E + i) * E;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int j = lane + 64 * q;
      if (j >= E) continue;
      const double ah = mx > 0.0 ? arow[j] * inv : 0.0;
      double task = 0.0;
      for (int f = 0; f < F; ++f) task += P[f * E + i] * P[f * E + j];
      const double at = (1.0 - alpha) * ah + alpha * (task * ah);
      const int64_t o = (static_cast<int64_t>(l) * E + i) * E + j;
      a_tilde[o] = static_cast<float>(at);
      if (a_hat) a_hat[o] = static_cast<float>(ah);
    }
  }
}

// GESR identification scores (Sec. 3.4, eq. generic-score) per row i of layer l, float64:
// Cent = sum_j A-bar(i, j); Cons = mean_f cos(A_f(i, :), A-bar(i, :)) (0 for a zero row);
// Spec = max_f ||A_f(i, :) - A-bar(i, :)||_2.  One wave per row, lanes over columns; the family rows
// are read twice (once for A-bar, once for the per-family terms), eight families' rows in flight at a
// time.  grid (L, row blocks), 256 threads.
__global__ __launch_bounds__(256) void gesr_scores_kernel(const uint32_t* __restrict__ D,
                                                          const uint32_t* __restrict__ C, int F, int L, int E, int k,
                                                          double* __restrict__ cent, double* __restrict__ cons,
                                                          double* __restrict__ spec) {
  __shared__ double inv_n[TACG_MAX_FAMILIES];
  const int l = blockIdx.x;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, nw = blockDim.x >> 6;
  // N_f of the layer: one wave per family, an exact integer sum over the experts
  for (int f = wave; f < F; f += nw) {
    const uint32_t* d = D + (static_cast<int64_t>(f) * L + l) * E;
    unsigned long long t = 0;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int e = lane + 64 * q;
      if (e < E) t += d[e];
    }
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) t += __shfl_xor(t, o, 64);
    const double n = static_cast<double>(t) / k;
    if (lane == 0) inv_n[f] = n > 0 ? 1.0 / n : 0.0;
  }
  __syncthreads();
  const int r0 = blockIdx.y * kRows, r1 = min(E, r0 + kRows);
  // the rows of families f0 .. f0 + 7 of row i (family index clamped into range)
  auto load_rows = [&](int i, int f0, uint32_t (&v)[kFamChunk][4]) {
#pragma unroll
    for (int u = 0; u < kFamChunk; ++u) {
      const int f = min(f0 + u, F - 1);
      const uint32_t* row = C + ((static_cast<int64_t>(f) * L + l) * E + i) * E;
#pragma unroll
      for (int q = 0; q < 4; ++q) v[u][q] = row[min(lane + 64 * q, E - 1)];
    }
  };
  for (int i = r0 + wave; i < r1; i += nw) {
    double ab[4] = {0, 0, 0, 0};
    for (int f0 = 0; f0 < F; f0 += kFamChunk) {
      uint32_t v[kFamChunk][4];
      load_rows(i, f0, v);
#pragma unroll
      for (int u = 0; u < kFamChunk; ++u) {
        const int f = f0 + u;
        if (f >= F) break;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int j = lane + 64 * q;
          if (j < E && j != i) ab[q] += v[u][q] * inv_n[f];
        }
      }
    }
    double cs = 0.0, nb2 = 0.0;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      ab[q] /= F;
      cs += ab[q];
      nb2 += ab[q] * ab[q];
    }
    cs = wave_sum(cs);
    nb2 = wave_sum(nb2);
    const double nb = sqrt(nb2);
    double cos_sum = 0.0, worst = 0.0;
    for (int f0 = 0; f0 < F; f0 += kFamChunk) {
      uint32_t v[kFamChunk][4];
      load_rows(i, f0, v);
#pragma unroll
      for (int u = 0; u < kFamChunk; ++u) {
        const int f = f0 + u;
        if (f >= F) break;
        double dot = 0.0, na2 = 0.0, dev2 = 0.0;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int j = lane + 64 * q;
          if (j < E) {
            const double a = (j != i) ? v[u][q] * inv_n[f] : 0.0;
            dot += a * ab[q];
            na2 += a * a;
            dev2 += (a - ab[q]) * (a - ab[q]);
          }
        }
        dot = wave_sum(dot);
        na2 = wave_sum(na2);
        dev2 = wave_sum(dev2);
        const double na = sqrt(na2);
        cos_sum += (na > 0.0 && nb > 0.0) ? dot / (na * nb) : 0.0;
        worst = fmax(worst, sqrt(dev2));
      }
    }
    if (lane == 0) {
      const int64_t o = static_cast<int64_t>(l) * E + i;
      cent[o] = cs;
      cons[o] = cos_sum / F;
      spec[o] = worst;
    }
  }
}

}  // namespace

size_t reweight_workspace(int32_t F, int32_t L, int32_t E) {
  size_t used = 0;
  carve_rw(nullptr, F, L, E, &used);
  return used;
}

int launch_reweight(const uint32_t* D, const uint32_t* C, int32_t F, int32_t L, int32_t E, int32_t k,
                    double alpha, double tau, double eps, float* pref, float* a_tilde, float* a_hat,
                    void* workspace, hipStream_t stream) {
  RwWs ws = carve_rw(workspace, F, L, E);
  const int rb = (E + kRows - 1) / kRows;
  const size_t plds = static_cast<size_t>(F) * E * sizeof(double);  // <= 64 x 256 x 8 = 128 KB
  hipLaunchKernelGGL(rw_nf, dim3(L, F), dim3(64), 0, stream, D, F, L, E, k, ws);
  hipLaunchKernelGGL(rw_rows, dim3(L, rb), dim3(256), 0, stream, C, F, L, E, ws);
  hipLaunchKernelGGL(rw_z, dim3(L, F), dim3(256), 0, stream, D, F, L, E, k, tau, eps, ws);
  (void)hipFuncSetAttribute(reinterpret_cast<const void*>(&rw_graph), hipFuncAttributeMaxDynamicSharedMemorySize,
                            static_cast<int>(plds));
  hipLaunchKernelGGL(rw_graph, dim3(L, rb), dim3(256), plds, stream, F, L, E, alpha, pref, a_tilde, a_hat, ws);
  return hipGetLastError() == hipSuccess ? TACG_OK : TACG_E_DEVICE;
}

int launch_gesr_scores(const uint32_t* D, const uint32_t* C, int32_t F, int32_t L, int32_t E, int32_t k, double* cent,
                       double* cons, double* spec, hipStream_t stream) {
  hipLaunchKernelGGL(gesr_scores_kernel, dim3(L, (E + kRows - 1) / kRows), dim3(256), 0, stream, D, C, F, L, E, k,
                     cent, cons, spec);
  return hipGetLastError() == hipSuccess ? TACG_OK : TACG_E_DEVICE;
}

}  // namespace tacg
