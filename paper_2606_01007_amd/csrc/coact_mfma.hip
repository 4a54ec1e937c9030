// Co-activation counts of small expert counts (E <= 64) on the matrix cores.
//
// For the tokens of one (family, layer) segment, C = R^T R where R[t][e] = 1 when token t selected
// expert e (Sec. 3.3: C counts the tokens that chose both experts).  With E <= 64 the whole Gram
// matrix is at most 2 x 2 blocks of 32 x 32, and the int8 MFMA v_mfma_i32_32x32x32_i8 adds the
// products of 32 tokens per instruction; at E = 64, top-6 that is 6 matrix instructions per 64
// token-layers instead of 15 scattered LDS increments per token-layer.  Used for k >= 5, where it
// is faster than the histogram (coact.hip).
//
// Kernel design (gfx950): one wave per workgroup; W waves each take one contiguous range of the
// flattened token-layers x = l * N + t (the same split as the histogram kernel, so the partial slots
// and the reduction are shared).  The ids of the next four batches are in flight while one is
// counted.  Per batch of 64 token-layers (one per lane):
//   * every lane validates its token's ids (range, repeats) and writes a 1 byte at [id][lane] of a
//     wave-private LDS tile [64 experts][64 tokens] (row stride 80 bytes, so that the 16-byte fragment
//     reads of eight consecutive lanes cover all 32 banks);
//   * for each half of the batch (32 tokens), lane l reads the 16 bytes of expert 32 i + l % 32 for
//     tokens 16 (l / 32) .. + 15 of that half: this one fragment is both the A operand (rows of R^T)
//     and the B operand (columns of R) of block i, since the k-th byte of a lane's A and B operands
//     stand for the same token;
//   * the blocks (0, 0), (0, 1) and (1, 1) accumulate in 32-bit registers ((1, 0) is the transpose);
//   * the bytes are cleared again by the same lanes.
// At a segment boundary the wave writes the strict upper triangle of its counts into partial slot
// w + s (every bin, so no clearing is needed) and starts again from zero.
#include "tacg_internal.h"

namespace tacg {
namespace {

typedef int v4i __attribute__((ext_vector_type(4)));
typedef int v16i __attribute__((ext_vector_type(16)));

constexpr int kRow = 80;                 // bytes per expert row of the tile (64 tokens + padding)
constexpr int kTile = 64 * kRow;         // bytes of the wave's tile

struct MfmaArgs {
  const int16_t* trace;
  int64_t N;
  int64_t total;
  int32_t L, E, F, W;
  int32_t nbins;
  uint32_t* partial;
  uint32_t* d_err;
  int64_t fam_off[TACG_MAX_FAMILIES + 1];
};

__device__ __forceinline__ uint32_t tri_bin(uint32_t m, uint32_t n, uint32_t E) {  // m < n
  return m * (2u * E - 3u - m) / 2u - 1u + n;
}

// Write the strict upper triangle of one 32 x 32 accumulator block (bi, bj).  Accumulator register r
// of lane l holds row 8 (r / 4) + 4 (l / 32) + r % 4 and column l % 32 of the block.
__device__ __forceinline__ void store_block(const v16i& acc, int bi, int bj, int lane, uint32_t E,
                                            uint32_t* __restrict__ dst) {
  const uint32_t n = 32u * bj + (lane & 31);
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    const uint32_t m = 32u * bi + 8u * (r >> 2) + 4u * (lane >> 5) + (r & 3);
    if (m < n && n < E) dst[tri_bin(m, n, E)] = static_cast<uint32_t>(acc[r]);
  }
}

// The raw ids of one token-layer (k int16 values), fetched ahead of their use.
template <int K>
struct Raw {
  uint16_t v[K];
  __device__ __forceinline__ void fetch(const int16_t* __restrict__ p) {
#pragma unroll
    for (int s = 0; s < K; ++s) v[s] = static_cast<uint16_t>(__builtin_nontemporal_load(p + s));
  }
};

constexpr int kDepth = 4;  // batches of ids in flight per lane

template <int K, int NB>
__global__ __launch_bounds__(64) void coact_mfma_kernel(MfmaArgs a) {
  __shared__ __align__(16) uint8_t tile[kTile];
  const int lane = threadIdx.x;
  const uint32_t E = static_cast<uint32_t>(a.E);
  // clear the tile once; afterwards every batch clears the bytes it set
  for (int i = lane * 16; i < kTile; i += 64 * 16) *reinterpret_cast<v4i*>(tile + i) = v4i{0, 0, 0, 0};
  __syncthreads();

  const int64_t w = blockIdx.x;
  int64_t pos = (w * a.total) / a.W;
  const int64_t end = ((w + 1) * a.total) / a.W;
  uint32_t err = 0;
  // this lane's fragment offsets: expert row 32 i + lane % 32, tokens 16 (lane / 32) .. + 15
  const int frag0 = (lane & 31) * kRow + 16 * (lane >> 5);

  while (pos < end) {
    const int64_t l = pos / a.N;
    const int64_t t0 = pos - l * a.N;
    int f = 0;
    while (a.fam_off[f + 1] <= t0) ++f;
    const int64_t stop = min(end, l * a.N + a.fam_off[f + 1]);
    const int64_t last = stop - 1;
    v16i acc00 = {}, acc01 = {}, acc11 = {};
    // ids of the next kDepth batches in flight; fetch addresses are clamped to the segment's last
    // token-layer, so every load is in bounds and the loop is uniform
    Raw<K> ring[kDepth];
#pragma unroll
    for (int d = 0; d < kDepth; ++d) {
      ring[d].fetch(a.trace + min(pos + 64 * d + lane, last) * K);
      __builtin_amdgcn_sched_barrier(0);
    }
    for (int64_t xb = pos; xb < stop; xb += 64 * kDepth) {
#pragma unroll
      for (int d = 0; d < kDepth; ++d) {
        const int64_t x = xb + 64 * d + lane;
        uint32_t ids[K];
        bool use = false;
        {
          unsigned long long seen = 0;
          bool ok = true, dup = false;
#pragma unroll
          for (int s = 0; s < K; ++s) {
            const uint32_t id = ring[d].v[s];  // negative ids became >= 32768 >= E
            ok &= id < E;
            const unsigned long long bit = 1ull << (id & 63u);
            dup |= (seen & bit) != 0ull;
            seen |= bit;
            ids[s] = id;
          }
          if (x < stop) {
            if (!ok) err |= TACG_ERR_ID_RANGE;
            else if (dup) err |= TACG_ERR_ID_DUP;
            use = ok && !dup;  // an invalid token-layer is flagged and not counted
          }
        }
        ring[d].fetch(a.trace + min(x + 64 * kDepth, last) * K);
        if (xb + 64 * d < stop) {  // batch-uniform: skip the matrix work of batches past the segment end
          if (use) {
#pragma unroll
            for (int s = 0; s < K; ++s) tile[ids[s] * kRow + lane] = 1;
          }
          __syncthreads();
#pragma unroll
          for (int h = 0; h < 2; ++h) {  // the two halves of 32 tokens
            const v4i f0 = *reinterpret_cast<const v4i*>(tile + frag0 + 32 * h);
            acc00 = __builtin_amdgcn_mfma_i32_32x32x32_i8(f0, f0, acc00, 0, 0, 0);
            if constexpr (NB == 2) {
              const v4i f1 = *reinterpret_cast<const v4i*>(tile + 32 * kRow + frag0 + 32 * h);
              acc01 = __builtin_amdgcn_mfma_i32_32x32x32_i8(f0, f1, acc01, 0, 0, 0);
              acc11 = __builtin_amdgcn_mfma_i32_32x32x32_i8(f1, f1, acc11, 0, 0, 0);
            }
          }
          __syncthreads();
          if (use) {
#pragma unroll
            for (int s = 0; s < K; ++s) tile[ids[s] * kRow + lane] = 0;
          }
        }
      }
    }
    uint32_t* dst = a.partial + (w + l * a.F + f) * static_cast<int64_t>(a.nbins);
    store_block(acc00, 0, 0, lane, E, dst);
    if constexpr (NB == 2) {
      store_block(acc01, 0, 1, lane, E, dst);
      store_block(acc11, 1, 1, lane, E, dst);
    }
    pos = stop;
  }
  if (err) atomicOr(a.d_err, err);
}

template <int K>
void launch_k(const MfmaArgs& a, hipStream_t stream) {
  if (a.E <= 32) hipLaunchKernelGGL((coact_mfma_kernel<K, 1>), dim3(a.W), dim3(64), 0, stream, a);
  else hipLaunchKernelGGL((coact_mfma_kernel<K, 2>), dim3(a.W), dim3(64), 0, stream, a);
}

}  // namespace

// The matrix path costs about the same at any k, the histogram k (k - 1) / 2 LDS increments per
// token-layer: measured on MI355X, 0.243 ms against 0.373 ms at E = 64, top-6 (2^21 tokens x 27
// layers), but 0.265 ms against 0.209 ms at E = 60, top-4 (3 x 2^20 tokens x 24 layers).
bool coact_uses_mfma(int32_t n_experts, int32_t top_k) { return n_experts <= 64 && top_k >= 5; }

int coact_mfma_workgroups(int64_t total) {
  // one wave per workgroup; about 8192 token-layers each, at most 4096 waves (16 per CU)
  const int64_t want = (total + 8191) / 8192;
  return static_cast<int>(std::max<int64_t>(1, std::min<int64_t>(4096, want)));
}

int launch_coact_mfma_hist(const int16_t* trace, int64_t n_tokens, int32_t n_layers, int32_t top_k,
                           int32_t n_experts, const int64_t* fam_off_host, int32_t n_fam, int32_t W, int32_t nbins,
                           uint32_t* partial, uint32_t* d_err, hipStream_t stream) {
  MfmaArgs a{};
  a.trace = trace;
  a.N = n_tokens;
  a.total = n_tokens * n_layers;
  a.L = n_layers;
  a.E = n_experts;
  a.F = n_fam;
  a.W = W;
  a.nbins = nbins;
  a.partial = partial;
  a.d_err = d_err;
  for (int f = 0; f <= n_fam; ++f) a.fam_off[f] = fam_off_host[f];
  switch (top_k) {
#define TACG_K(k)             \
  case k:                     \
    launch_k<k>(a, stream);   \
    break;
    TACG_K(2) TACG_K(3) TACG_K(4) TACG_K(5) TACG_K(6) TACG_K(7) TACG_K(8)
    TACG_K(9) TACG_K(10) TACG_K(11) TACG_K(12) TACG_K(13) TACG_K(14) TACG_K(15) TACG_K(16)
#undef TACG_K
    default:
      return TACG_E_UNSUPPORTED;
  }
  return hipGetLastError() == hipSuccess ? TACG_OK : TACG_E_DEVICE;
}

}  // namespace tacg
