// Dispatch and co-activation counts per (family, layer) segment of an int16 routing trace.
//
// Counting (Sec. 3.3: u and A of family f at layer l are frequencies over f's tokens):
//   D[f][l][i] = #tokens choosing i,  C[f][l][i][j] = #tokens choosing both i and j (i != j).
//
// Kernel design (gfx950):
//   * The trace is flattened to token-layers x = l * N + t.  Segments (l, f) are contiguous ranges of
//     x, so W persistent workgroups each take one contiguous range [x0, x1) and walk the segments it
//     crosses.  One thread per token-layer; the k ids are read with one 16/8/4-byte vector load.
//   * Each workgroup keeps a private upper-triangle histogram of the E(E-1)/2 expert pairs in LDS
//     (uint32, 130,560 B at E = 256, so one workgroup per CU).  The k ids are sorted in registers by
//     a Batcher odd-even merge network; then pair (x_i, x_j), i < j, lives at triangle index
//     T = x_i (2E - 3 - x_i) / 2 - 1 + x_j, so every pair costs one address add and one ds_add_u32.
//     The diagonal is not counted: each valid token with expert i adds exactly k - 1 pairs to row i,
//     so D_i = (sum_j C_ij) / (k - 1) is recovered exactly in the reduction.
//   * At every segment boundary the workgroup stores its histogram into partial slot (w + s) of the
//     workspace (slot indices are unique because both w and s grow along x), then zeroes it.
//   * A second kernel, one workgroup per segment, sums the partial slots of the workgroups that
//     touched the segment and writes the dense symmetric C (diagonal = D) and D.
#include "tacg_internal.h"

namespace tacg {
namespace {

struct CoactArgs {
  const int16_t* trace;
  int64_t N;           // tokens
  int64_t total;       // L * N token-layers
  int32_t L, K, E, F;
  int32_t W;           // workgroups of the histogram kernel
  int32_t nbins;       // histogram bins per slot
  uint32_t* partial;   // [(W + L * F)][nbins]
  uint32_t* d_err;
  int64_t fam_off[TACG_MAX_FAMILIES + 1];
};

__device__ __forceinline__ void cmp_swap(uint32_t& a, uint32_t& b) {
  const uint32_t lo = min(a, b), hi = max(a, b);
  a = lo;
  b = hi;
}

// Batcher odd-even merge sort of n = 2^m values (fully unrolled; comparisons against padding
// constants fold away).
template <int NP2>
__device__ __forceinline__ void sort_network(uint32_t* v) {
#pragma unroll
  for (int p = 1; p < NP2; p <<= 1) {
#pragma unroll
    for (int k = p; k >= 1; k >>= 1) {
#pragma unroll
      for (int j = k % p; j + k < NP2; j += 2 * k) {
#pragma unroll
        for (int i = 0; i < k; ++i) {
          if (i + j + k < NP2 && (i + j) / (2 * p) == (i + j + k) / (2 * p)) cmp_swap(v[i + j], v[i + j + k]);
        }
      }
    }
  }
}

constexpr int next_pow2(int k) { return k <= 1 ? 1 : 2 * next_pow2((k + 1) / 2); }

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

// The k ids of one token-layer as unsigned 16-bit values (negative ids become >= 32768 >= E).
template <int K>
__device__ __forceinline__ void load_ids(const int16_t* __restrict__ p, uint32_t* x) {
  if constexpr (K % 8 == 0) {
#pragma unroll
    for (int q = 0; q < K / 8; ++q) {
      const u32x4 v = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p) + q);
      const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        x[8 * q + 2 * r] = w[r] & 0xffffu;
        x[8 * q + 2 * r + 1] = w[r] >> 16;
      }
    }
  } else if constexpr (K % 4 == 0) {
#pragma unroll
    for (int q = 0; q < K / 4; ++q) {
      const u32x2 v = __builtin_nontemporal_load(reinterpret_cast<const u32x2*>(p) + q);
      x[4 * q] = v.x & 0xffffu;
      x[4 * q + 1] = v.x >> 16;
      x[4 * q + 2] = v.y & 0xffffu;
      x[4 * q + 3] = v.y >> 16;
    }
  } else if constexpr (K % 2 == 0) {
#pragma unroll
    for (int q = 0; q < K / 2; ++q) {
      const uint32_t v = __builtin_nontemporal_load(reinterpret_cast<const uint32_t*>(p) + q);
      x[2 * q] = v & 0xffffu;
      x[2 * q + 1] = v >> 16;
    }
  } else {
#pragma unroll
    for (int q = 0; q < K; ++q) x[q] = static_cast<uint16_t>(p[q]);
  }
}

template <int K>
__global__ __launch_bounds__(kCoactThreads) void coact_hist_kernel(CoactArgs a) {
  extern __shared__ uint32_t hist[];
  constexpr int NP2 = next_pow2(K);
  const int tid = threadIdx.x;
  const int nb = a.nbins;
  for (int i = tid; i < nb; i += blockDim.x) hist[i] = 0u;
  __syncthreads();

  const int64_t w = blockIdx.x;
  int64_t pos = (w * a.total) / a.W;
  const int64_t end = ((w + 1) * a.total) / a.W;
  const uint32_t E = static_cast<uint32_t>(a.E);
  const uint32_t rbk = 2u * (2u * E - 3u);
  uint32_t err = 0;

  while (pos < end) {
    const int64_t l = pos / a.N;
    const int64_t t = pos - l * a.N;
    int f = 0;
    while (a.fam_off[f + 1] <= t) ++f;
    const int64_t stop = min(end, l * a.N + a.fam_off[f + 1]);
    for (int64_t x = pos + tid; x < stop; x += blockDim.x) {
      uint32_t v[NP2];
      load_ids<K>(a.trace + x * K, v);
#pragma unroll
      for (int i = K; i < NP2; ++i) v[i] = 0xffffu;
      if constexpr (K == 1) {
        if (v[0] < E) {
          __hip_atomic_fetch_add(&hist[v[0]], 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
        } else {
          err |= TACG_ERR_ID_RANGE;
        }
      } else {
        sort_network<NP2>(v);
        bool dup = false;
#pragma unroll
        for (int i = 0; i + 1 < K; ++i) dup |= (v[i] == v[i + 1]);
        const bool range_bad = v[K - 1] >= E;
        if (dup | range_bad) {
          err |= (range_bad ? TACG_ERR_ID_RANGE : 0u) | (dup ? TACG_ERR_ID_DUP : 0u);
        } else {
          // byte offset of the triangle row of each id taken as the smaller member of a pair
          uint32_t rb[K - 1];
#pragma unroll
          for (int i = 0; i < K - 1; ++i) rb[i] = v[i] * (rbk - 2u * v[i]) - 4u;
#pragma unroll
          for (int i = 0; i < K - 1; ++i) {
#pragma unroll
            for (int j = i + 1; j < K; ++j) {
              uint32_t* cell = reinterpret_cast<uint32_t*>(__builtin_assume_aligned(
                  reinterpret_cast<char*>(hist) + (rb[i] + 4u * v[j]), 4));
              __hip_atomic_fetch_add(cell, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
            }
          }
        }
      }
    }
    __syncthreads();
    uint32_t* dst = a.partial + (w + l * a.F + f) * static_cast<int64_t>(nb);
    for (int i = tid; i < nb; i += blockDim.x) {
      dst[i] = hist[i];
      hist[i] = 0u;
    }
    __syncthreads();
    pos = stop;
  }
  if (err) atomicOr(a.d_err, err);
}

// Workgroup whose range [x0(w), x1(w)) contains token-layer x.
__device__ __forceinline__ int64_t owner_of(int64_t x, int64_t total, int64_t W) {
  return ((x + 1) * W + total - 1) / total - 1;
}

// One workgroup per segment s = l * F + f.  Each wave takes rows i; lanes take columns j.
__global__ __launch_bounds__(256) void coact_reduce_kernel(CoactArgs a, uint32_t* __restrict__ D,
                                                           uint32_t* __restrict__ C, uint32_t accumulate) {
  const int s = blockIdx.x;
  const int l = s / a.F, f = s % a.F;
  const int E = a.E;
  const int64_t seg0 = static_cast<int64_t>(l) * a.N + a.fam_off[f];
  const int64_t seg1 = static_cast<int64_t>(l) * a.N + a.fam_off[f + 1];
  int64_t w0 = 1, w1 = 0;  // no contributors for an empty segment
  if (seg1 > seg0) {
    w0 = owner_of(seg0, a.total, a.W);
    w1 = owner_of(seg1 - 1, a.total, a.W);
  }
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int nwaves = blockDim.x >> 6;
  uint32_t* Dseg = D + (static_cast<int64_t>(f) * a.L + l) * E;
  uint32_t* Cseg = C + (static_cast<int64_t>(f) * a.L + l) * E * static_cast<int64_t>(E);
  const int64_t nb = a.nbins;

  for (int i = wave; i < E; i += nwaves) {
    uint32_t rowsum = 0;
    for (int j = lane; j < E; j += 64) {
      uint32_t v = 0;
      if (a.K == 1) {
        if (j == i)
          for (int64_t w = w0; w <= w1; ++w) v += a.partial[(w + s) * nb + i];
      } else if (j != i) {
        const uint32_t lo = min(i, j), hi = max(i, j);
        const uint32_t T = lo * (2u * E - 3u - lo) / 2u - 1u + hi;
        for (int64_t w = w0; w <= w1; ++w) v += a.partial[(w + s) * nb + T];
        rowsum += v;
      }
      if (j != i) {
        uint32_t* c = Cseg + static_cast<int64_t>(i) * E + j;
        *c = accumulate ? *c + v : v;
      } else if (a.K == 1) {
        rowsum = v;
      }
    }
    // wave reduction of the row sum -> D_i
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) rowsum += __shfl_xor(rowsum, o, 64);
    if (lane == 0) {
      const uint32_t d = (a.K == 1) ? rowsum : rowsum / static_cast<uint32_t>(a.K - 1);
      uint32_t* c = Cseg + static_cast<int64_t>(i) * E + i;
      const uint32_t dn = accumulate ? Dseg[i] + d : d;
      Dseg[i] = dn;
      *c = dn;
    }
  }
}

template <int K>
void launch_hist(const CoactArgs& a, size_t lds, hipStream_t stream) {
  (void)hipFuncSetAttribute(reinterpret_cast<const void*>(&coact_hist_kernel<K>),
                      hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(lds));
  hipLaunchKernelGGL(coact_hist_kernel<K>, dim3(a.W), dim3(kCoactThreads), lds, stream, a);
}

}  // namespace

size_t coact_bins(int32_t n_experts, int32_t top_k) {
  if (top_k == 1) return static_cast<size_t>(n_experts);
  return static_cast<size_t>(n_experts) * static_cast<size_t>(n_experts - 1) / 2;
}

int coact_num_workgroups(int64_t total, int32_t n_experts) {
  // one workgroup per CU when the triangle needs more than half of the 160 KB LDS, else two
  const int64_t cap = (n_experts > 128) ? 256 : 512;
  const int64_t want = (total + 32767) / 32768;
  return static_cast<int>(std::max<int64_t>(1, std::min(cap, want)));
}

int launch_coact(const int16_t* trace, int64_t n_tokens, int32_t n_layers, int32_t top_k, int32_t n_experts,
                 const int64_t* fam_off_host, int32_t n_fam, uint32_t* D, uint32_t* C, uint32_t flags,
                 uint32_t* d_err, void* workspace, hipStream_t stream) {
  CoactArgs a{};
  a.trace = trace;
  a.N = n_tokens;
  a.total = n_tokens * n_layers;
  a.L = n_layers;
  a.K = top_k;
  a.E = n_experts;
  a.F = n_fam;
  a.W = coact_num_workgroups(a.total, n_experts);
  a.nbins = static_cast<int32_t>(coact_bins(n_experts, top_k));
  a.partial = static_cast<uint32_t*>(workspace);
  a.d_err = d_err;
  for (int f = 0; f <= n_fam; ++f) a.fam_off[f] = fam_off_host[f];
  const size_t lds = static_cast<size_t>(a.nbins) * sizeof(uint32_t);
  if (a.total > 0) {
    switch (top_k) {
#define TACG_K(k) \
  case k:         \
    launch_hist<k>(a, lds, stream); \
    break;
      TACG_K(1) TACG_K(2) TACG_K(3) TACG_K(4) TACG_K(5) TACG_K(6) TACG_K(7) TACG_K(8)
      TACG_K(9) TACG_K(10) TACG_K(11) TACG_K(12) TACG_K(13) TACG_K(14) TACG_K(15) TACG_K(16)
#undef TACG_K
      default:
        return TACG_E_UNSUPPORTED;
    }
    if (hipGetLastError() != hipSuccess) return TACG_E_DEVICE;
  }
  if (a.total == 0) a.total = 1;  // the reduction sees no contributors (all segments empty)
  hipLaunchKernelGGL(coact_reduce_kernel, dim3(n_layers * n_fam), dim3(256), 0, stream, a, D, C,
                     (flags & TACG_ACCUMULATE) ? 1u : 0u);
  if (hipGetLastError() != hipSuccess) return TACG_E_DEVICE;
  return TACG_OK;
}

}  // namespace tacg
