// Co-activation counts of small expert counts (E <= 128) on the matrix cores.
//
// For the tokens of one (family, layer) segment, C = R^T R where R[t][e] = 1 when token t selected
// expert e (Sec. 3.3: C counts the tokens that chose both experts).  With E <= 32 NB the Gram matrix
// has NB x NB blocks of 32 x 32 (NB = 1, 2 or 4); v_mfma_f32_32x32x64_f8f6f4 with 4-bit (e2m1)
// operands adds the products of 64 tokens per instruction, so 64 token-layers cost NB (NB + 1) / 2
// matrix instructions (the blocks on and above the diagonal: 3 at E <= 64, 10 at E <= 128),
// whatever k is.
//
// Kernel design (gfx950): one wave per workgroup; W waves each take one contiguous range of the
// flattened token-layers x = l * N + t (the split of the histogram kernel, so the partial slots and
// the reduction are shared).  The ids of the next four batches are in flight while one is counted.
// Per batch of 64 token-layers (one per lane):
//   * each lane forms its token's one-hot row in registers: a 64-bit mask of its ids (128-bit at
//     NB = 4, where bit 6 of the id picks the 64-bit half), which also validates them: a repeated
//     id leaves fewer than k bits, an id of E or more sets a bit outside the lane's valid set or a
//     bit above bit 5 (bit 6 at NB = 4) of its raw word.  The mask is turned into one e2m1 nibble
//     per expert (0x1 = 0.5, so a product is 0.25 and every float32 partial sum is exact).  The nibbles
//     come from byte permutes used as a four-entry table: selector byte j = two mask bits, output
//     byte j = those two bits as two nibbles, so a row of 32 experts costs four permutes, four ANDs
//     and three shifts.  For that, row position n holds the mask bit relabel(n), where relabel
//     swaps bit fields 4:3 and 2:1 of the index (an involution that keeps bits 5 and 6, so every
//     32-expert block keeps its experts); the Gram matrix is thus counted over relabelled experts
//     and mapped back when the triangle is written;
//   * the lane stores the row (16 NB bytes, token-major) into a wave-private LDS tile with 16-byte
//     writes.  The 8-byte chunks of a row (16 experts each) sit at positions permuted by the row
//     number (chunk c of row j at c ^ s(j)), which makes the reads below bank-conflict-free, and
//     the lanes whose rows share banks write their 16-byte parts in different orders (part q ^ g(j)
//     in store q), which makes the stores conflict-free; both permutations are XOR constants per
//     lane (relabelled like the ids), applied to the ids before the mask is formed, so they cost
//     nothing per token;
//   * ds_read_b64_tr_b4 reads 16 rows x 16 nibbles per group of 16 lanes and hands lane i the
//     nibbles of column i: two such reads give lane l the 32 nibbles of expert 32 b + l % 32 over
//     tokens 32 (l / 32) .. + 31 of the batch.  That fragment is both the A operand (row of R^T) and
//     the B operand (column of R) of block b, since the j-th nibble of a lane's A and B operands
//     stands for the same token; the product is exact whatever the hardware's k order.
// No clearing is needed (every row is overwritten), and two tiles alternate, so a wave's writes of
// one batch never meet its reads of the previous one.  The LDS executes one wave's instructions in
// order, so the reads see the same wave's preceding writes without a barrier.
// At a segment boundary the wave writes the strict upper triangle of its counts into partial slot
// w + s (every bin, so no clearing is needed) and starts again from zero.
#include "tacg_internal.h"

namespace tacg {
namespace {

typedef int v2i __attribute__((ext_vector_type(2)));
typedef int v4i __attribute__((ext_vector_type(4)));
typedef int v8i __attribute__((ext_vector_type(8)));
typedef float v16f __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kFmtFp4 = 4;  // operand format code of the f8f6f4 matrix instructions: e2m1

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
// of lane l holds row 8 (r / 4) + 4 (l / 32) + r % 4 and column l % 32 of the block, as 0.25 x count;
// row and column positions are relabelled experts.
// Expert index <-> row position (see the file comment): swap bits 4:3 with bits 2:1.
__device__ __forceinline__ uint32_t relabel(uint32_t x) {
  return (x & 0x61u) | ((x & 0x18u) >> 2) | ((x & 0x06u) << 2);
}

// Mask-bit permutations that XOR-ing the bit index with 4, 32 or 64 applies to a 128-bit mask held
// as two 64-bit halves.
__device__ __forceinline__ uint64_t swap_nibbles(uint64_t x) {
  return ((x & 0x0f0f0f0f0f0f0f0full) << 4) | ((x >> 4) & 0x0f0f0f0f0f0f0f0full);
}
__device__ __forceinline__ uint64_t swap_dwords(uint64_t x) { return (x << 32) | (x >> 32); }

__device__ __forceinline__ void store_block(const v16f& acc, int bi, int bj, int lane, uint32_t E,
                                            uint32_t* __restrict__ dst) {
  const uint32_t n = 32u * bj + (lane & 31);
  const uint32_t en = relabel(n);
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    const uint32_t m = 32u * bi + 8u * (r >> 2) + 4u * (lane >> 5) + (r & 3);
    const uint32_t em = relabel(m);
    if (m < n && em < E && en < E) dst[tri_bin(min(em, en), max(em, en), E)] = static_cast<uint32_t>(acc[r] * 4.0f);
  }
}

// The raw ids of one token-layer, fetched ahead of their use (k int16 values; dword loads for even k).
template <int K>
struct Raw {
  static constexpr int kWords = (K % 2 == 0) ? K / 2 : K;
  uint32_t w[kWords];
  __device__ __forceinline__ void fetch(const int16_t* __restrict__ p) {
    if constexpr (K % 2 == 0) {
#pragma unroll
      for (int q = 0; q < kWords; ++q) w[q] = __builtin_nontemporal_load(reinterpret_cast<const uint32_t*>(p) + q);
    } else {
#pragma unroll
      for (int q = 0; q < kWords; ++q) w[q] = static_cast<uint16_t>(__builtin_nontemporal_load(p + q));
    }
  }
  __device__ __forceinline__ uint32_t any_id_bits() const {  // OR of the raw words
    uint32_t o = 0;
#pragma unroll
    for (int q = 0; q < kWords; ++q) o |= w[q];
    return o;
  }
  __device__ __forceinline__ uint32_t id(int s) const {  // negative ids become >= 32768 >= E
    if constexpr (K % 2 == 0) return (s & 1) ? (w[s >> 1] >> 16) : (w[s >> 1] & 0xffffu);
    else return w[s];
  }
};

// Byte permute as a table lookup: selector byte j in 0..3 picks byte j of {0x00, 0x01, 0x10, 0x11},
// so two mask bits (bits 0 and 1 of selector byte j) become two nibbles of value 1 in output byte j.
__device__ __forceinline__ uint32_t nibble_pairs(uint32_t sel, uint32_t keep) {
  return __builtin_amdgcn_perm(0u, 0x11100100u, sel & keep);
}

constexpr int kDepth = 4;  // batches of ids in flight per lane (even: steps alternate the two tiles)

// Add one batch's products: the blocks (bi, bj), bi <= bj, of the Gram matrix, in row order (fp4
// operands in the low four registers of each 8-register operand).
template <int NB>
__device__ __forceinline__ void mfma_blocks(const v4i (&frag)[NB], v16f (&acc)[NB * (NB + 1) / 2]) {
  v8i f[NB];
#pragma unroll
  for (int b = 0; b < NB; ++b) f[b] = v8i{frag[b].x, frag[b].y, frag[b].z, frag[b].w, 0, 0, 0, 0};
  int b = 0;
#pragma unroll
  for (int bi = 0; bi < NB; ++bi) {
#pragma unroll
    for (int bj = bi; bj < NB; ++bj, ++b)
      acc[b] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(f[bi], f[bj], acc[b], kFmtFp4, kFmtFp4, 0, 0, 0, 0);
  }
}

constexpr int log2i(int x) { return x <= 1 ? 0 : 1 + log2i(x / 2); }

// NB = number of 32-expert blocks (1: E <= 32, 2: E <= 64, 4: E <= 128).  The register budget is set
// for four waves per SIMD (the three accumulator blocks of NB = 2 take 48 registers), two at NB = 4
// (ten blocks, 160 registers).
template <int K, int NB>
__global__ __launch_bounds__(64) __attribute__((amdgpu_waves_per_eu(NB == 4 ? 2 : 4, 8))) void coact_mfma_kernel(
    MfmaArgs a) {
  static_assert(NB == 1 || NB == 2 || NB == 4, "one, two or four 32-expert blocks");
  constexpr int kMaskWords = NB == 4 ? 4 : 2;  // 32-bit words of the id mask (ids below 32 kMaskWords)
  constexpr int kRowBytes = 16 * NB;                 // 4-bit one-hot row of 32 NB experts
  constexpr int kChunks = 2 * NB;                    // 8-byte chunks (16 experts) per row
  constexpr int kSwShift = log2i(128 / kRowBytes);   // s(j) = (j >> kSwShift) & (kChunks - 1)
  constexpr int kPartShift = log2i(8 / NB);          // g(j) = (j >> kPartShift) & (NB - 1)
  constexpr int kBlocks = NB * (NB + 1) / 2;
  constexpr int kTileBytes = 64 * kRowBytes;
  __shared__ __align__(16) uint8_t tile[2 * kTileBytes];
  const int lane = threadIdx.x;
  const uint32_t E = static_cast<uint32_t>(a.E);

  const int64_t w = blockIdx.x;
  int64_t pos = (w * a.total) / a.W;
  const int64_t end = ((w + 1) * a.total) / a.W;
  uint32_t err = 0;

  // this lane's row (token lane of the batch): the physical chunk of logical chunk c is c ^ s(j);
  // store q writes the row's 16-byte part q ^ g(j), so register chunk slot t holds physical chunk
  // t ^ 2 g(j), i.e. logical chunk t ^ 2 g(j) ^ s(j): the ids are XOR-ed with that constant
  const uint32_t sw_row = (static_cast<uint32_t>(lane) >> kSwShift) & (kChunks - 1);
  const uint32_t part_row = (static_cast<uint32_t>(lane) >> kPartShift) & (NB - 1);
  const uint32_t id_xor = relabel((sw_row ^ (part_row << 1)) << 4);
  // mask bits b whose expert b ^ id_xor is >= E (id_xor has bits 2, 5 and 6 only)
  uint32_t nv[kMaskWords];
  {
    uint64_t lo = E >= 64u ? 0ull : (~0ull << E);
    uint64_t hi = E >= 128u ? 0ull : (E <= 64u ? ~0ull : (~0ull << (E - 64u)));
    if (id_xor & 4u) {
      lo = swap_nibbles(lo);
      hi = swap_nibbles(hi);
    }
    if (id_xor & 32u) {
      lo = swap_dwords(lo);
      hi = swap_dwords(hi);
    }
    if (id_xor & 64u) {
      const uint64_t t = lo;
      lo = hi;
      hi = t;
    }
    nv[0] = static_cast<uint32_t>(lo);
    nv[1] = static_cast<uint32_t>(lo >> 32);
    if constexpr (kMaskWords == 4) {
      nv[2] = static_cast<uint32_t>(hi);
      nv[3] = static_cast<uint32_t>(hi >> 32);
    }
  }
  const uint32_t row_off = static_cast<uint32_t>(lane) * kRowBytes;
  // transposed reads: lane l = 16 g + i reads, for block b and half r, the chunk of experts
  // 32 b + 16 (g & 1) .. + 15 of row j = 32 (g >> 1) + 16 r + i
  uint32_t rd_off[NB][2];
  {
    const int g = lane >> 4, i = lane & 15;
#pragma unroll
    for (int b = 0; b < NB; ++b) {
#pragma unroll
      for (int r = 0; r < 2; ++r) {
        const uint32_t j = 32u * (g >> 1) + 16u * r + i;
        const uint32_t c = 2u * b + (g & 1);
        const uint32_t p = c ^ ((j >> kSwShift) & (kChunks - 1));
        rd_off[b][r] = j * kRowBytes + 8u * p;
      }
    }
  }
  // LDS byte offset of the tile: the low 32 bits of a generic address into the LDS aperture
  const uint32_t tile_base = static_cast<uint32_t>(reinterpret_cast<uintptr_t>(tile));

  while (pos < end) {
    const int64_t l = pos / a.N;
    const int64_t t0 = pos - l * a.N;
    int f = 0;
    while (a.fam_off[f + 1] <= t0) ++f;
    const int64_t stop = min(end, l * a.N + a.fam_off[f + 1]);
    // this wave's part of the segment, addressed with 32-bit offsets from a uniform pointer (the
    // host keeps every wave's range below 2^24 token-layers, for the 24-bit offset products)
    const int16_t* __restrict__ segp = a.trace + pos * K;
    const uint32_t n = static_cast<uint32_t>(stop - pos);
    const uint32_t nlast = n - 1u;
    v16f acc[kBlocks];
#pragma unroll
    for (int b = 0; b < kBlocks; ++b) acc[b] = v16f{};
    // ids of the next kDepth batches in flight; fetch offsets are clamped to the last token-layer,
    // so every load is in bounds and the loop is uniform
    Raw<K> ring[kDepth];
#pragma unroll
    for (int d = 0; d < kDepth; ++d) {
      ring[d].fetch(segp + __umul24(min(static_cast<uint32_t>(64 * d + lane), nlast), static_cast<uint32_t>(K)));
      __builtin_amdgcn_sched_barrier(0);
    }
    // software pipeline: the transposed reads of batch i are issued right after its rows are
    // stored, and its matrix instructions run only after batch i + 1's rows are built, so the VALU
    // work of the next batch covers the read latency.  Step d of the unrolled loop always uses tile
    // d % 2 (kDepth is even), so all LDS addresses are fixed.
    bool have = false;  // frag holds the fragments of a batch whose products are still to be added
    v4i frag[NB];
    for (uint32_t rb = 0; rb < n; rb += 64 * kDepth) {
#pragma unroll
      for (int d = 0; d < kDepth; ++d) {
        const uint32_t base = rb + 64u * d;  // batch-uniform
        // one-hot mask of the ids (the 64-bit shift uses the low six bits of its amount; at NB = 4
        // bit 6 picks the 64-bit half)
        uint32_t mw[kMaskWords];
        if constexpr (kMaskWords == 2) {
          uint64_t m = 0;
#pragma unroll
          for (int s = 0; s < K; ++s) m |= 1ull << ((ring[d].id(s) ^ id_xor) & 63u);
          mw[0] = static_cast<uint32_t>(m);
          mw[1] = static_cast<uint32_t>(m >> 32);
        } else {
#pragma unroll
          for (int i = 0; i < kMaskWords; ++i) mw[i] = 0u;
#pragma unroll
          for (int s = 0; s < K; ++s) {
            const uint32_t b = ring[d].id(s) ^ id_xor;
            const uint64_t t = 1ull << (b & 63u);
            const uint32_t t0 = static_cast<uint32_t>(t), t1 = static_cast<uint32_t>(t >> 32);
            const uint32_t hs = static_cast<uint32_t>(__builtin_amdgcn_sbfe(static_cast<int>(b), 6, 1));
            mw[0] = __builtin_amdgcn_bitop3_b32(mw[0], t0, hs, 0xF4);  // mw | (t & ~hs)
            mw[1] = __builtin_amdgcn_bitop3_b32(mw[1], t1, hs, 0xF4);
            mw[2] = __builtin_amdgcn_bitop3_b32(mw[2], t0, hs, 0xF8);  // mw | (t & hs)
            mw[3] = __builtin_amdgcn_bitop3_b32(mw[3], t1, hs, 0xF8);
          }
        }
        const bool in_seg = lane < static_cast<int>(n - base);
        // raw ids of 64 (128 at NB = 4) or more, then mask bits of experts >= E
        uint32_t oor = ring[d].any_id_bits() & (NB == 4 ? 0xff80ff80u : 0xffc0ffc0u);
        int pop = 0;
#pragma unroll
        for (int i = 0; i < kMaskWords; ++i) {
          oor |= mw[i] & nv[i];
          pop += __popc(mw[i]);
        }
        const bool range_bad = oor != 0u;
        const bool dup = pop != K;
        err |= (in_seg && range_bad) ? TACG_ERR_ID_RANGE : 0u;
        err |= (in_seg && !range_bad && dup) ? TACG_ERR_ID_DUP : 0u;
        // an invalid token-layer is flagged and not counted
        const uint32_t keep = (!in_seg || range_bad || dup) ? 0u : 0x03030303u;
        ring[d].fetch(reinterpret_cast<const int16_t*>(reinterpret_cast<const char*>(segp) +
                      __umul24(min(lane + (base + 64u * kDepth), nlast), static_cast<uint32_t>(2 * K))));
        const bool active = base < n;  // batch-uniform
        const uint32_t kBuf = (d & 1) * kTileBytes;
        if (active) {
          uint8_t* rowp = tile + kBuf + row_off;
#pragma unroll
          for (int q = 0; q < NB; ++q) {  // register part q (32 experts) to the row's part q ^ g(j)
            const uint32_t src = mw[q];
            u32x4 v;
            v.x = nibble_pairs(src, keep);
            v.y = nibble_pairs(src >> 2, keep);
            v.z = nibble_pairs(src >> 4, keep);
            v.w = nibble_pairs(src >> 6, keep);
            *reinterpret_cast<u32x4*>(rowp + 16 * (q ^ part_row)) = v;
          }
        }
        if (have) mfma_blocks<NB>(frag, acc);  // the previous batch
        have = false;
        if (active) {
          // the reads address the tile through raw LDS offsets the compiler cannot relate to the
          // stores above: keep them in program order (the LDS then executes them in order)
          __asm__ __volatile__("" ::: "memory");
#pragma unroll
          for (int b = 0; b < NB; ++b) {
            const v2i r0 = __builtin_amdgcn_ds_read_tr4_b64_v2i32(
                (__attribute__((address_space(3))) v2i*)(uintptr_t)(tile_base + kBuf + rd_off[b][0]));
            const v2i r1 = __builtin_amdgcn_ds_read_tr4_b64_v2i32(
                (__attribute__((address_space(3))) v2i*)(uintptr_t)(tile_base + kBuf + rd_off[b][1]));
            frag[b] = v4i{r0.x, r0.y, r1.x, r1.y};
          }
          __asm__ __volatile__("" ::: "memory");
          have = true;
        }
      }
    }
    if (have) mfma_blocks<NB>(frag, acc);
    uint32_t* dst = a.partial + (w + l * a.F + f) * static_cast<int64_t>(a.nbins);
    // the bin addresses depend only on the lane: an opaque copy of E keeps the compiler from
    // hoisting all 48 of them out of the segment loop into registers
    uint32_t Es = E;
    __asm__ __volatile__("" : "+s"(Es));
    // likewise an opaque copy of the lane for the relabelled bin indices
    int ln = lane;
    __asm__ __volatile__("" : "+v"(ln));
    {
      int b = 0;
#pragma unroll
      for (int bi = 0; bi < NB; ++bi) {
#pragma unroll
        for (int bj = bi; bj < NB; ++bj) store_block(acc[b++], bi, bj, ln, Es, dst);
      }
    }
    pos = stop;
  }
  if (err) atomicOr(a.d_err, err);
}

template <int K>
void launch_k(const MfmaArgs& a, hipStream_t stream) {
  if (a.E <= 32) hipLaunchKernelGGL((coact_mfma_kernel<K, 1>), dim3(a.W), dim3(64), 0, stream, a);
  else if (a.E <= 64) hipLaunchKernelGGL((coact_mfma_kernel<K, 2>), dim3(a.W), dim3(64), 0, stream, a);
  else hipLaunchKernelGGL((coact_mfma_kernel<K, 4>), dim3(a.W), dim3(64), 0, stream, a);
}

}  // namespace

// The matrix path costs about the same at any k, the histogram k (k - 1) / 2 LDS increments per
// token-layer (coact.hip).  Measured on MI355X (kernel averages): at E = 64, top-6 (2^21 tokens x 27
// layers) 143 us against 0.37 ms for the histogram; at E = 60, top-4 (2^22 tokens x 24 layers) 164 us
// against 184 us.  The four-block kernel (E <= 128; ten products per 64 token-layers, 160 accumulator
// registers, two waves per SIMD) costs twice the two-block one per token-layer, so it pays only from
// top-8, timed per call on 2^21 tokens x 24 layers at E = 128: 0.365 against 0.376 ms at top-8 with
// uniform ids, 0.384 against 0.305 ms at top-7, 0.349 against 0.244 ms at top-6; on the clustered
// E = 128, top-8 trace of 2^22 tokens x 48 layers 1.18 against 1.43 ms.  Above top-12 its register
// budget spills, so the histogram keeps those.
bool coact_uses_mfma(int32_t n_experts, int32_t top_k) {
  return (n_experts <= 64 && top_k >= 4) || (n_experts <= 128 && top_k >= 8 && top_k <= 12);
}

int coact_mfma_workgroups(int64_t total, int32_t n_experts) {
  // one wave per workgroup; about 8192 token-layers each, at most 16 waves per CU at E <= 64 and 8
  // at E <= 128 (all resident)
  const int64_t cap = n_experts <= 64 ? 4096 : 2048;
  const int64_t want = (total + 8191) / 8192;
  return static_cast<int>(std::max<int64_t>(1, std::min<int64_t>(cap, want)));
}

int launch_coact_mfma_hist(const int16_t* trace, int64_t n_tokens, int32_t n_layers, int32_t top_k,
                           int32_t n_experts, const int64_t* fam_off_host, int32_t n_fam, int32_t W, int32_t nbins,
                           uint32_t* partial, uint32_t* d_err, hipStream_t stream) {
  // each wave addresses its range with 24-bit products of token-layer offsets: keep it below 2^24
  // token-layers (at least 2048 waves when the range is long, so this holds for any trace below 2^35
  // token-layers)
  if ((n_tokens * n_layers + W - 1) / W >= (int64_t(1) << 24)) return TACG_E_UNSUPPORTED;
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
