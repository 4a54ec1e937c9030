// Motivation diagnostics of App. H (auxiliary metrics) from the co-activation counts:
//   * activation Frobenius distance between the expert-activation distributions of two families,
//     P_f[l][e] = D_f[l][e] / N_{f,l}, dist[i][j] = ||P_i - P_j||_F over all layers and experts;
//   * top-n co-activated pair sets per (family, layer) and their Jaccard overlaps per layer.
//
// dist_kernel: one workgroup per family pair, one wave per layer (wave sums only), float64.
// top_pairs_kernel: one workgroup per (family, layer).  The segment's upper triangle is staged in
//   LDS (130,560 B at E = 256; rows by waves, coalesced), the n-th largest positive count T is found by bisection on counts,
//   pairs above T are kept, ties at T are kept in increasing pair order until n are chosen (a
//   chunked block scan gives each tie its rank), and the chosen pairs are written in increasing pair
//   order (a second scan gives each its slot).
// jaccard_kernel: one wave per (layer, family pair); every element of one sorted list is looked up
//   in the other by bisection.
#include "tacg_internal.h"

namespace tacg {
namespace {

constexpr int kDistThreads = 256;
constexpr int kTopThreads = 1024;

__device__ __forceinline__ double wave_sum_d(double v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

// sum over the workgroup of 64-bit unsigned values; every thread gets the result
__device__ unsigned long long block_sum_u64(unsigned long long v, unsigned long long* red) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o, 64);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, nw = blockDim.x >> 6;
  __syncthreads();
  if (lane == 0) red[wave] = v;
  __syncthreads();
  unsigned long long t = 0;
  for (int i = 0; i < nw; ++i) t += red[i];
  return t;
}

// exclusive prefix sum over the workgroup of one value per thread (in thread order)
__device__ uint32_t block_exclusive_scan(uint32_t v, uint32_t* buf, uint32_t& total) {
  const int t = threadIdx.x, n = blockDim.x;
  __syncthreads();
  buf[t] = v;
  __syncthreads();
  for (int off = 1; off < n; off <<= 1) {  // Hillis-Steele inclusive scan
    const uint32_t add = (t >= off) ? buf[t - off] : 0u;
    __syncthreads();
    buf[t] += add;
    __syncthreads();
  }
  total = buf[n - 1];
  return buf[t] - v;
}

__global__ __launch_bounds__(kDistThreads) void dist_kernel(const uint32_t* __restrict__ D, int F, int L, int E, int k,
                                                            double* __restrict__ dist) {
  __shared__ double dred[kDistThreads / 64];
  const int i = blockIdx.x, j = blockIdx.y;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, nw = blockDim.x >> 6;
  double acc = 0.0;
  for (int l = wave; l < L; l += nw) {  // one wave per layer, lanes over experts
    const uint32_t* Di = D + (static_cast<int64_t>(i) * L + l) * E;
    const uint32_t* Dj = D + (static_cast<int64_t>(j) * L + l) * E;
    uint32_t di[4], dj[4];
    unsigned long long si = 0, sj = 0;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int e = lane + 64 * q;
      di[q] = e < E ? Di[e] : 0u;
      dj[q] = e < E ? Dj[e] : 0u;
      si += di[q];
      sj += dj[q];
    }
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) {
      si += __shfl_xor(si, o, 64);
      sj += __shfl_xor(sj, o, 64);
    }
    // P = D / N with N = sum_e D / k, i.e. P = k * D / sum_e D (0 for an empty family)
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const double pi = si ? static_cast<double>(di[q]) / (static_cast<double>(si) / k) : 0.0;
      const double pj = sj ? static_cast<double>(dj[q]) / (static_cast<double>(sj) / k) : 0.0;
      acc += (pi - pj) * (pi - pj);
    }
  }
  acc = wave_sum_d(acc);
  if (lane == 0) dred[wave] = acc;
  __syncthreads();
  if (threadIdx.x == 0) {
    double s = 0.0;
    for (int w = 0; w < nw; ++w) s += dred[w];
    dist[static_cast<int64_t>(i) * F + j] = sqrt(s);
  }
}

// triangle index of pair (a, b), a < b, in row-major order of the strict upper triangle
__device__ __forceinline__ uint32_t tri_index(uint32_t a, uint32_t b, uint32_t E) {
  return a * (2u * E - a - 1u) / 2u + (b - a - 1u);
}

__global__ __launch_bounds__(kTopThreads) void top_pairs_kernel(const uint32_t* __restrict__ C, int F, int L, int E,
                                                                int top_n, int32_t* __restrict__ out) {
  extern __shared__ uint32_t tri[];
  __shared__ unsigned long long red[kTopThreads / 64];
  __shared__ uint32_t scan[kTopThreads];
  const int f = blockIdx.x, l = blockIdx.y;
  const int tid = threadIdx.x, nt = blockDim.x;
  const uint32_t UE = static_cast<uint32_t>(E);
  const uint32_t npairs = UE * (UE - 1u) / 2u;
  const uint32_t* seg = C + (static_cast<int64_t>(f) * L + l) * E * static_cast<int64_t>(E);
  // stage the strict upper triangle row by row: each wave takes rows, lanes take columns; four rows
  // per step, all their loads in flight (addresses clamped into the segment, stores only for a < b)
  {
    const int lane = tid & 63, wave = tid >> 6, nw = nt >> 6;
    for (int a0 = wave; a0 < E; a0 += 4 * nw) {
      uint32_t v[4][4];
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int a = min(a0 + r * nw, E - 1);
#pragma unroll
        for (int q = 0; q < 4; ++q) v[r][q] = seg[a * E + min(a + 1 + lane + 64 * q, E - 1)];
      }
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int a = a0 + r * nw;
        if (a < E) {
          const uint32_t base = tri_index(static_cast<uint32_t>(a), static_cast<uint32_t>(a) + 1u, UE);
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            const int b = a + 1 + lane + 64 * q;
            if (b < E) tri[base + static_cast<uint32_t>(b - a - 1)] = v[r][q];
          }
        }
      }
    }
  }
  __syncthreads();
  // this thread's contiguous chunk of the triangle; an odd chunk length puts the 32 threads of a
  // half-wave on 32 different LDS banks at every step of the chunk scans
  const uint32_t per = ((npairs + nt - 1) / nt) | 1u;
  const uint32_t t0 = min(npairs, tid * per), t1 = min(npairs, t0 + per);
  // largest count
  uint32_t mx = 0;
  for (uint32_t t = t0; t < t1; ++t) mx = max(mx, tri[t]);
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) mx = max(mx, __shfl_xor(mx, o, 64));
  __syncthreads();
  if ((tid & 63) == 0) scan[tid >> 6] = mx;
  __syncthreads();
  mx = 0;
  for (int w = 0; w < nt / 64; ++w) mx = max(mx, scan[w]);
  // T = the largest threshold >= 1 with at least top_n pairs at or above it (1 if fewer exist)
  auto count_ge = [&](uint32_t T) {
    unsigned long long c = 0;
    for (uint32_t t = t0; t < t1; ++t) c += tri[t] >= T;
    return block_sum_u64(c, red);
  };
  uint32_t lo = 1, hi = max(mx, 1u);  // count_ge(lo) >= top_n or lo == 1; search the largest such T
  while (lo < hi) {
    const uint32_t mid = lo + (hi - lo + 1u) / 2u;
    if (count_ge(mid) >= static_cast<unsigned long long>(top_n)) lo = mid;
    else hi = mid - 1u;
  }
  const uint32_t T = lo;
  const unsigned long long above = count_ge(T + 1u);
  const uint32_t need = static_cast<uint32_t>(
      min(static_cast<unsigned long long>(top_n), count_ge(T)) - min(above, static_cast<unsigned long long>(top_n)));
  // rank of every tie (count == T) in pair order
  uint32_t ties = 0;
  for (uint32_t t = t0; t < t1; ++t) ties += tri[t] == T;
  uint32_t total;
  uint32_t rank = block_exclusive_scan(ties, scan, total);
  // chosen pairs of this chunk, then their slots in pair order
  uint32_t chosen = 0;
  for (uint32_t t = t0; t < t1; ++t) {
    const uint32_t c = tri[t];
    if (c > T || (c == T && rank < need)) ++chosen;
    if (c == T) ++rank;
  }
  uint32_t n_chosen;
  uint32_t slot = block_exclusive_scan(chosen, scan, n_chosen);
  int32_t* dst = out + (static_cast<int64_t>(f) * L + l) * top_n;
  rank = rank - ties;  // back to this chunk's first tie rank
  if (t0 < t1) {
    // (a, b) of the chunk's first pair, then walk the row-major triangle
    uint32_t a = 0;
    while (tri_index(a, UE - 1u, UE) < t0) ++a;
    uint32_t b = t0 - tri_index(a, a + 1u, UE) + a + 1u;
    for (uint32_t t = t0; t < t1; ++t) {
      const uint32_t c = tri[t];
      const bool take = c > T || (c == T && rank < need);
      if (c == T) ++rank;
      if (take && slot < static_cast<uint32_t>(top_n)) dst[slot++] = static_cast<int32_t>(a * UE + b);
      if (++b == UE) {
        ++a;
        b = a + 1u;
      }
    }
  }
  for (int s = static_cast<int>(n_chosen) + tid; s < top_n; s += nt) dst[s] = -1;
}

// number of entries >= 0 of a list padded with -1
__device__ __forceinline__ int list_len(const int32_t* v, int n) {
  int lo = 0, hi = n;  // first index holding -1 (the valid entries come first)
  while (lo < hi) {
    const int mid = (lo + hi) / 2;
    if (v[mid] >= 0) lo = mid + 1;
    else hi = mid;
  }
  return lo;
}

__global__ __launch_bounds__(64) void jaccard_kernel(const int32_t* __restrict__ pairs, int F, int L, int top_n,
                                                     double* __restrict__ jac) {
  const int l = blockIdx.x, i = blockIdx.y, j = blockIdx.z;
  const int32_t* a = pairs + (static_cast<int64_t>(i) * L + l) * top_n;
  const int32_t* b = pairs + (static_cast<int64_t>(j) * L + l) * top_n;
  const int na = list_len(a, top_n), nb = list_len(b, top_n);
  int inter = 0;
  for (int q = threadIdx.x; q < na; q += 64) {
    const int32_t x = a[q];
    int lo = 0, hi = nb;
    while (lo < hi) {
      const int mid = (lo + hi) / 2;
      if (b[mid] < x) lo = mid + 1;
      else hi = mid;
    }
    inter += (lo < nb && b[lo] == x) ? 1 : 0;
  }
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) inter += __shfl_xor(inter, o, 64);
  if (threadIdx.x == 0) {
    const int uni = na + nb - inter;
    jac[(static_cast<int64_t>(l) * F + i) * F + j] = uni ? static_cast<double>(inter) / uni : 1.0;
  }
}

}  // namespace

int launch_activation_distance(const uint32_t* D, int32_t F, int32_t L, int32_t E, int32_t k, double* dist,
                               hipStream_t stream) {
  hipLaunchKernelGGL(dist_kernel, dim3(F, F), dim3(kDistThreads), 0, stream, D, F, L, E, k, dist);
  return hipGetLastError() == hipSuccess ? TACG_OK : TACG_E_DEVICE;
}

int launch_pair_jaccard(const uint32_t* C, int32_t F, int32_t L, int32_t E, int32_t top_n, int32_t* top_pairs,
                        double* jaccard, hipStream_t stream) {
  const size_t lds = static_cast<size_t>(E) * (E - 1) / 2 * sizeof(uint32_t);
  (void)hipFuncSetAttribute(reinterpret_cast<const void*>(&top_pairs_kernel),
                            hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(lds));
  hipLaunchKernelGGL(top_pairs_kernel, dim3(F, L), dim3(kTopThreads), lds, stream, C, F, L, E, top_n, top_pairs);
  hipLaunchKernelGGL(jaccard_kernel, dim3(L, F, F), dim3(64), 0, stream, top_pairs, F, L, top_n, jaccard);
  return hipGetLastError() == hipSuccess ? TACG_OK : TACG_E_DEVICE;
}

}  // namespace tacg
