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
//   * At E <= 64 with k >= 4, and at E <= 128 with 8 <= k <= 12, the partial slots come from 4-bit
//     matrix products instead (coact_mfma.hip), with the same split of x, the same slots and the
//     same reduction.
#include "tacg_internal.h"

namespace tacg {
namespace {

constexpr int kReduceThreads = 1024;
constexpr int kCoactSmallE = 128;        // at most this many experts: the small-triangle launch
constexpr int kCoactThreadsLarge = 1024;  // threads per histogram workgroup, E > kCoactSmallE
constexpr int kCoactThreadsSmall = 512;   // threads per histogram workgroup, E <= kCoactSmallE
constexpr int kDepth = 4;  // token-layers per thread in flight in coact_hist_kernel

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

// The raw k ids of one token-layer, fetched with the widest aligned loads (rows of k int16 are
// 2k bytes, so even k allows 4-, 8- or 16-byte loads), and unpacked to unsigned 16-bit values
// (negative ids become >= 32768 >= E).  Fetch and unpack are separate so that the next token-layer's
// loads are in flight while the current one is counted.
template <int K>
struct RawIds {
  static constexpr int kWords = (K % 2 == 0) ? K / 2 : K;  // dwords (even k) or halfwords (odd k)
  uint32_t w[kWords];

  __device__ __forceinline__ void fetch(const int16_t* __restrict__ p) {
    if constexpr (K % 8 == 0) {
#pragma unroll
      for (int q = 0; q < K / 8; ++q) {
        const u32x4 v = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p) + q);
        w[4 * q] = v.x;
        w[4 * q + 1] = v.y;
        w[4 * q + 2] = v.z;
        w[4 * q + 3] = v.w;
      }
    } else if constexpr (K % 4 == 0) {
#pragma unroll
      for (int q = 0; q < K / 4; ++q) {
        const u32x2 v = __builtin_nontemporal_load(reinterpret_cast<const u32x2*>(p) + q);
        w[2 * q] = v.x;
        w[2 * q + 1] = v.y;
      }
    } else if constexpr (K % 2 == 0) {
#pragma unroll
      for (int q = 0; q < K / 2; ++q) w[q] = __builtin_nontemporal_load(reinterpret_cast<const uint32_t*>(p) + q);
    } else {
#pragma unroll
      for (int q = 0; q < K; ++q) w[q] = static_cast<uint16_t>(p[q]);
    }
  }

  __device__ __forceinline__ void unpack(uint32_t* x) const {
    if constexpr (K % 2 == 0) {
#pragma unroll
      for (int q = 0; q < K / 2; ++q) {
        x[2 * q] = w[q] & 0xffffu;
        x[2 * q + 1] = w[q] >> 16;
      }
    } else {
#pragma unroll
      for (int q = 0; q < K; ++q) x[q] = w[q];
    }
  }
};

constexpr uint64_t kOddLanes = 0xaaaaaaaaaaaaaaaaull;  // lanes with bit 0 set
constexpr uint64_t kLaneBit1 = 0xccccccccccccccccull;  // lanes with bit 1 set

// Per-lane choice from a wave-uniform lane mask: b in the lanes whose mask bit is set, else a.
__device__ __forceinline__ uint32_t lane_select(uint32_t a, uint32_t b, uint64_t lanes) {
  uint32_t r;
  asm("v_cndmask_b32 %0, %1, %2, %3" : "=v"(r) : "v"(a), "v"(b), "s"(lanes));
  return r;
}

// Count one token-layer into the workgroup's triangle (see the file comment).
template <int K>
__device__ __forceinline__ void count_token(const RawIds<K>& raw, bool valid, uint32_t* hist, uint32_t E,
                                            uint32_t& err) {
  constexpr int NP2 = next_pow2(K);
  uint32_t v[NP2];
  raw.unpack(v);
#pragma unroll
  for (int i = K; i < NP2; ++i) v[i] = 0xffffu;
  if constexpr (K == 1) {
    if (valid) {
      if (v[0] < E) {
        __hip_atomic_fetch_add(&hist[v[0]], 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
      } else {
        err |= TACG_ERR_ID_RANGE;
      }
    }
  } else {
    sort_network<NP2>(v);
    bool dup = false;
#pragma unroll
    for (int i = 0; i + 1 < K; ++i) dup |= (v[i] == v[i + 1]);
    const bool range_bad = v[K - 1] >= E;
    if (valid && (dup | range_bad)) {
      err |= (range_bad ? TACG_ERR_ID_RANGE : 0u) | (dup ? TACG_ERR_ID_DUP : 0u);
    } else if (valid) {
      // byte offset of the triangle row of each id taken as the smaller member of a pair:
      // 4 * (x (2E - 3 - x) / 2 - 1) = x (2 (2E - 3) - 2x) - 4; both factors fit 24 bits
      const uint32_t rbk = 2u * (2u * E - 3u);
      uint32_t rb[K - 1];
#pragma unroll
      for (int i = 0; i < K - 1; ++i) rb[i] = __umul24(v[i], rbk - 2u * v[i]) - 4u;
      if constexpr (K >= 6 && K <= 8) {
        // Lanes walk their pair lists in one of four orders (lane bit 0: reversed, bit 1: rotated by
        // half the list).  A pair that is frequent in a family tends to sit at the same place in the
        // sorted pair lists of many tokens, and lanes that add to one address in the same instruction
        // are serialised; the four orders split those collisions.  Measured on MI355X at top-8 against
        // one order: 1.68 -> 1.42 ms at E = 128 (48 layers x 2^22 tokens), 3.38 -> 3.16 ms at E = 256;
        // eight orders gained nothing more, and at top-4 the selects cost more than they save.
        constexpr int NP = K * (K - 1) / 2;
        uint32_t off[NP];
        int n = 0;
#pragma unroll
        for (int i = 0; i < K - 1; ++i) {
#pragma unroll
          for (int j = i + 1; j < K; ++j) off[n++] = rb[i] + 4u * v[j];
        }
        if constexpr (K == 8) {
          const bool rev = (threadIdx.x & 1u) != 0u;
          const bool rot = (threadIdx.x & 2u) != 0u;
#pragma unroll
          for (int q = 0; q < NP; ++q) {
            const int q2 = (q + NP / 2) % NP;
            const uint32_t x = rev ? off[NP - 1 - q] : off[q];
            const uint32_t y = rev ? off[NP - 1 - q2] : off[q2];
            uint32_t* cell = reinterpret_cast<uint32_t*>(__builtin_assume_aligned(
                reinterpret_cast<char*>(hist) + (rot ? y : x), 4));
            __hip_atomic_fetch_add(cell, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
          }
        } else {
          // At top-6 and top-7 the plain selects above were turned into selects of array indices
          // and then into chains of selects (about 220 and 430 select instructions per token-layer
          // instead of 36 and 48; 2.5x and 3.5x slower at E = 256).  Here the selects take
          // their lane masks from constant SGPR pairs, two per pair.  At top-8 the compiler keeps
          // two selects per pair by itself, and its schedule measured 0.7 % faster.
          uint32_t x[NP];
#pragma unroll
          for (int q = 0; q < NP; ++q) x[q] = lane_select(off[q], off[NP - 1 - q], kOddLanes);
#pragma unroll
          for (int q = 0; q < NP; ++q) {
            uint32_t* cell = reinterpret_cast<uint32_t*>(__builtin_assume_aligned(
                reinterpret_cast<char*>(hist) + lane_select(x[q], x[(q + NP / 2) % NP], kLaneBit1), 4));
            __hip_atomic_fetch_add(cell, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
          }
        }
      } else {
#pragma unroll
        for (int i = 0; i < K - 1; ++i) {
#pragma unroll
          for (int j = i + 1; j < K; ++j) {
            uint32_t* cell = reinterpret_cast<uint32_t*>(
                __builtin_assume_aligned(reinterpret_cast<char*>(hist) + (rb[i] + 4u * v[j]), 4));
            __hip_atomic_fetch_add(cell, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
          }
        }
      }
    }
  }
}

template <int K, int THREADS>
__global__ __launch_bounds__(THREADS) void coact_hist_kernel(CoactArgs a) {
  extern __shared__ uint32_t hist[];
  const int tid = threadIdx.x;
  const int nb = a.nbins;
  for (int i = tid; i < nb; i += blockDim.x) hist[i] = 0u;
  __syncthreads();

  const int64_t w = blockIdx.x;
  int64_t pos = (w * a.total) / a.W;
  const int64_t end = ((w + 1) * a.total) / a.W;
  const uint32_t E = static_cast<uint32_t>(a.E);
  uint32_t err = 0;

  while (pos < end) {
    const int64_t l = pos / a.N;
    const int64_t t = pos - l * a.N;
    int f = 0;
    while (a.fam_off[f + 1] <= t) ++f;
    const int64_t stop = min(end, l * a.N + a.fam_off[f + 1]);
    // one token-layer per thread and step.  The ids of the next kDepth - 1 steps are in flight in
    // a ring of buffers while one step is counted; fetch addresses are clamped to the segment's last
    // token-layer, so every load is unconditional and in bounds, and the loop is workgroup-uniform
    // (a thread past the end of the segment fetches and sorts but does not count).
    const int64_t bd = blockDim.x, last = stop - 1;
    RawIds<K> ring[kDepth];
#pragma unroll
    for (int d = 0; d < kDepth; ++d) {
      ring[d].fetch(a.trace + min(pos + tid + d * bd, last) * K);
      // keep the issue order ring[0], ring[1], ...: the loop below then waits for one buffer at a time
      __builtin_amdgcn_sched_barrier(0);
    }
    for (int64_t xb = pos; xb < stop; xb += kDepth * bd) {
#pragma unroll
      for (int d = 0; d < kDepth; ++d) {
        const int64_t x = xb + d * bd + tid;
        count_token<K>(ring[d], x < stop, hist, E, err);
        ring[d].fetch(a.trace + min(x + kDepth * bd, last) * K);
      }
    }
    barrier_after_lds_atomics();
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

// One workgroup per segment s = l * F + f.  The partial triangles of the workgroups that touched
// the segment are summed into LDS with coalesced reads; then each wave writes dense rows i of C
// (lanes over columns j, coalesced) from the LDS triangle and recovers D_i from the row sum.
// Both phases are branch-free in their inner loops (indices are clamped and the values selected),
// so every load of a thread is in flight before the first wait: one workgroup fills a CU, and the
// HBM latency has to be covered by the loads of its own threads.
template <bool ACC, int NQ>  // NQ = ceil(E / 64) columns per lane
__global__ __launch_bounds__(kReduceThreads) void coact_reduce_kernel(CoactArgs a, uint32_t* __restrict__ D,
                                                                      uint32_t* __restrict__ C) {
  extern __shared__ uint32_t tri[];
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
  const int nb = a.nbins;  // >= 1
  constexpr int kUnroll = 4 * NQ;  // about nbins / kReduceThreads loads per thread
  // slots summed per round: about 16 loads per thread in flight (many workgroups' slots meet in one
  // segment when each workgroup covers a short range, as on the matrix-core path)
  constexpr int kSlots = kUnroll >= 16 ? 1 : 16 / kUnroll;
  for (int b0 = threadIdx.x; b0 < nb; b0 += kUnroll * kReduceThreads) {
    uint32_t v[kUnroll] = {};
    for (int64_t w = w0; w <= w1; w += kSlots) {
      uint32_t x[kSlots][kUnroll];
#pragma unroll
      for (int j = 0; j < kSlots; ++j) {
        // slots past w1 are read clamped to w1 (in bounds) and then dropped
        const uint32_t* src = a.partial + (min(w + j, w1) + s) * static_cast<int64_t>(nb);
#pragma unroll
        for (int u = 0; u < kUnroll; ++u)
          x[j][u] = __builtin_nontemporal_load(src + min(b0 + u * kReduceThreads, nb - 1));
      }
#pragma unroll
      for (int j = 0; j < kSlots; ++j) {
        const uint32_t keep = (w + j <= w1) ? ~0u : 0u;
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) v[u] += x[j][u] & keep;
      }
    }
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const int b = b0 + u * kReduceThreads;
      if (b < nb) tri[b] = v[u];
    }
  }
  __syncthreads();

  const uint32_t lane = threadIdx.x & 63u;
  const int wave = threadIdx.x >> 6;
  constexpr int nwaves = kReduceThreads / 64;
  const uint32_t ue = static_cast<uint32_t>(E);
  const uint32_t rk = 2u * ue - 3u;
  const bool pairs = a.K > 1;
  uint32_t* Dseg = D + (static_cast<int64_t>(f) * a.L + l) * E;
  uint32_t* Cseg = C + (static_cast<int64_t>(f) * a.L + l) * E * static_cast<int64_t>(E);
  for (int i = wave; i < E; i += nwaves) {
    const uint32_t ui = static_cast<uint32_t>(i);
    uint32_t* crow = Cseg + static_cast<int64_t>(i) * E;
    uint32_t val[NQ];
    uint32_t rowsum = 0;
#pragma unroll
    for (int q = 0; q < NQ; ++q) {
      const uint32_t j = lane + 64u * q;
      const uint32_t lo = min(ui, j), hi = max(ui, j);
      const bool off = pairs && j < ue && j != ui;
      const uint32_t x = tri[off ? lo * (rk - lo) / 2u - 1u + hi : 0u];
      val[q] = off ? x : 0u;
      rowsum += val[q];
    }
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) rowsum += __shfl_xor(rowsum, o, 64);
    // each valid token with expert i adds k - 1 pairs to row i; with k = 1 the bins are D itself
    const uint32_t d = pairs ? rowsum / static_cast<uint32_t>(a.K - 1) : tri[i];
    const uint32_t dn = ACC ? Dseg[i] + d : d;
#pragma unroll
    for (int q = 0; q < NQ; ++q) {
      const uint32_t j = lane + 64u * q;
      if (j < ue) {
        uint32_t out = (j == ui) ? dn : val[q];
        if (ACC && j != ui) out += crow[j];
        crow[j] = out;
      }
    }
    if (lane == 0) Dseg[i] = dn;
  }
}

template <bool ACC, int NQ>
void launch_reduce_t(const CoactArgs& a, dim3 grid, size_t lds, uint32_t* D, uint32_t* C, hipStream_t stream) {
  (void)hipFuncSetAttribute(reinterpret_cast<const void*>(&coact_reduce_kernel<ACC, NQ>),
                            hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(lds));
  hipLaunchKernelGGL((coact_reduce_kernel<ACC, NQ>), grid, dim3(kReduceThreads), lds, stream, a, D, C);
}

template <bool ACC>
void launch_reduce(const CoactArgs& a, int nq, dim3 grid, size_t lds, uint32_t* D, uint32_t* C, hipStream_t stream) {
  static_assert(TACG_MAX_EXPERTS <= 4 * 64, "one to four column chunks per lane");
  switch (nq) {
    case 1: launch_reduce_t<ACC, 1>(a, grid, lds, D, C, stream); break;
    case 2: launch_reduce_t<ACC, 2>(a, grid, lds, D, C, stream); break;
    case 3: launch_reduce_t<ACC, 3>(a, grid, lds, D, C, stream); break;
    default: launch_reduce_t<ACC, 4>(a, grid, lds, D, C, stream); break;
  }
}

template <int K, int THREADS>
void launch_hist_t(const CoactArgs& a, size_t lds, hipStream_t stream) {
  (void)hipFuncSetAttribute(reinterpret_cast<const void*>(&coact_hist_kernel<K, THREADS>),
                            hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(lds));
  hipLaunchKernelGGL((coact_hist_kernel<K, THREADS>), dim3(a.W), dim3(THREADS), lds, stream, a);
}

template <int K>
void launch_hist(const CoactArgs& a, size_t lds, hipStream_t stream) {
  if (a.E > kCoactSmallE) launch_hist_t<K, kCoactThreadsLarge>(a, lds, stream);
  else launch_hist_t<K, kCoactThreadsSmall>(a, lds, stream);
}

}  // namespace

size_t coact_bins(int32_t n_experts, int32_t top_k) {
  if (top_k == 1) return static_cast<size_t>(n_experts);
  return static_cast<size_t>(n_experts) * static_cast<size_t>(n_experts - 1) / 2;
}

int coact_num_workgroups(int64_t total, int32_t n_experts, int32_t top_k) {
  if (coact_uses_mfma(n_experts, top_k)) return coact_mfma_workgroups(total, n_experts);
  // E > 128: the triangle needs more than half of the 160 KB LDS, so one 1024-thread workgroup per
  // CU; otherwise four 512-thread workgroups per CU (the same 32 waves, with four private triangles)
  const int64_t cap = (n_experts > kCoactSmallE) ? 256 : 1024;
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
  a.W = coact_num_workgroups(a.total, n_experts, top_k);
  a.nbins = static_cast<int32_t>(coact_bins(n_experts, top_k));
  a.partial = static_cast<uint32_t*>(workspace);
  a.d_err = d_err;
  for (int f = 0; f <= n_fam; ++f) a.fam_off[f] = fam_off_host[f];
  const size_t lds = static_cast<size_t>(a.nbins) * sizeof(uint32_t);
  if (a.total > 0 && coact_uses_mfma(n_experts, top_k)) {
    const int rc = launch_coact_mfma_hist(trace, n_tokens, n_layers, top_k, n_experts, fam_off_host, n_fam, a.W,
                                          a.nbins, a.partial, d_err, stream);
    if (rc != TACG_OK) return rc;
  } else if (a.total > 0) {
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
  const int nq = (n_experts + 63) / 64;
  if (flags & TACG_ACCUMULATE) {
    launch_reduce<true>(a, nq, dim3(n_layers * n_fam), lds, D, C, stream);
  } else {
    launch_reduce<false>(a, nq, dim3(n_layers * n_fam), lds, D, C, stream);
  }
  if (hipGetLastError() != hipSuccess) return TACG_E_DEVICE;
  return TACG_OK;
}

}  // namespace tacg
